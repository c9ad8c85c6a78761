// Prefix-based index grouping (FlowTT Section 3.3, Fig. 4) on gfx950:
//   ingest   -> one 32-bit key per occurrence, t*Npad + g (invalid rows get Npad*T)
//   sort     -> LSD radix sort of (key, position), 8-bit digits, stable
//   unique   -> row heads and prefix-group heads, counted per tile and scanned
//   RLE      -> unique rows, inverse map, occurrence ranges, prefix groups
//   order    -> prefix groups re-ordered (table, i2, i1) through a dense scan over
//               the prefix space, cut into work slices of at most SLICE_ROWS rows
// All kernels are plain HIP for wave64; no library sort or scan is used.
#include "common.h"

namespace ttemb {

// ---------------------------------------------------------------------------
// fills
// ---------------------------------------------------------------------------
__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = v;
}

hipError_t fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)blocks), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t fill_f32(float* p, int64_t n, float v, hipStream_t st) {
  union {
    float f;
    uint32_t u;
  } c;
  c.f = v;
  return fill_u32(reinterpret_cast<uint32_t*>(p), n, c.u, st);
}

// ---------------------------------------------------------------------------
// ingest: keys, positions and bag ids, one tile of SORT_TILE occurrences per block
// ---------------------------------------------------------------------------
constexpr int INGEST_WIN = SORT_TILE + 1;

__device__ __forceinline__ int64_t upper_bound_global(const int64_t* a, int64_t lo, int64_t hi, int64_t x) {
  // first index in [lo, hi) with a[i] > x (hi if none)
  while (lo < hi) {
    int64_t mid = lo + ((hi - lo) >> 1);
    if (a[mid] <= x)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

// tile_bag[k] = the bag whose occurrence range holds occurrence k * SORT_TILE
// (entries stay 0 where invalid offsets leave a tile start uncovered); also
// flags offsets that are not a CSR partition of [0, M) in the error word
__global__ void k_tile_bags(const int64_t* __restrict__ offsets, int64_t NB, int64_t M,
                            int32_t* __restrict__ tile_bag, int32_t* __restrict__ ctr) {
  const int64_t b = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (b >= NB) return;
  int64_t lo = offsets[b], hi = offsets[b + 1];
  if (lo < 0 || hi < lo || hi > M || (b == 0 && lo != 0) || (b == NB - 1 && hi != M))
    atomicOr(&ctr[C_ERR], ERR_OFFSETS);
  lo = lo < 0 ? 0 : (lo > M ? M : lo);
  hi = hi < lo ? lo : (hi > M ? M : hi);
  for (int64_t k = (lo + SORT_TILE - 1) / SORT_TILE; k * SORT_TILE < hi; ++k) tile_bag[k] = (int32_t)b;
}

__global__ void __launch_bounds__(SORT_THREADS) k_ingest(const int64_t* __restrict__ idx, int64_t M,
                                                         const int64_t* __restrict__ offsets,
                                                         const int32_t* __restrict__ tile_bag, int64_t B, int T,
                                                         int64_t N, uint32_t Npad, uint32_t kinv,
                                                         uint32_t* __restrict__ keys, uint32_t* __restrict__ vals,
                                                         int32_t* __restrict__ bag_of, int32_t* __restrict__ ctr,
                                                         uint32_t* __restrict__ counts0, int nb0, int ntiles) {
  __shared__ int64_t win[INGEST_WIN];
  __shared__ uint32_t h0[1 << RADIX_MAX_BITS];  // digit counts of the first sort pass (bits 0 .. log2 nb0)
  const int64_t NB = (int64_t)T * B;
  // tiles in order, an eighth per XCD, as the sort's first pass takes them: that pass
  // reads a tile's keys and positions on the XCD that wrote them
  const int tile = (int)xcd_block(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int64_t o0 = (int64_t)tile * SORT_TILE;
  const int64_t o1 = (o0 + SORT_TILE < M ? o0 + SORT_TILE : M);
  // every index of the thread's items is loaded before any is used, and before the
  // bag window, so the loads are in flight together
  int64_t gv[SORT_ITEMS];
#pragma unroll
  for (int j = 0; j < SORT_ITEMS; ++j) {
    const int64_t o = o0 + (int64_t)j * SORT_THREADS + threadIdx.x;
    gv[j] = o < o1 ? __builtin_nontemporal_load(idx + o) : 0;
  }
  if (counts0)
    for (int d = threadIdx.x; d < nb0; d += SORT_THREADS) h0[d] = 0u;
  int64_t bfirst = 0, nwin = 0;
  if (offsets) {
    // bags of this tile: from the bag holding o0 to the one holding the next tile's first occurrence
    int64_t f = tile_bag[tile];
    int64_t l = o1 < M ? (int64_t)tile_bag[tile + 1] : NB - 1;
    f = f < 0 ? 0 : (f > NB - 1 ? NB - 1 : f);
    l = l < f ? f : (l > NB - 1 ? NB - 1 : l);
    bfirst = f;
    nwin = l - f + 2;  // offsets[bfirst .. l + 1]
    if (nwin <= INGEST_WIN)
      for (int k = threadIdx.x; k < nwin; k += SORT_THREADS) win[k] = offsets[bfirst + k];
  }
  __syncthreads();  // the bag window and the cleared digit counts
  int err = 0;
#pragma unroll
  for (int j = 0; j < SORT_ITEMS; ++j) {
    const int64_t o = o0 + (int64_t)j * SORT_THREADS + threadIdx.x;
    if (o >= o1) break;
    int64_t b;
    if (!offsets) {
      b = o;
    } else if (nwin <= INGEST_WIN) {
      int lo = 0, hi = (int)nwin;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (win[mid] <= o)
          lo = mid + 1;
        else
          hi = mid;
      }
      b = bfirst + lo - 1;
    } else {
      b = upper_bound_global(offsets, 0, NB + 1, o) - 1;
    }
    b = b < 0 ? 0 : (b > NB - 1 ? NB - 1 : b);
    const int64_t g = gv[j];
    const uint32_t t = (uint32_t)b / (uint32_t)B;
    uint32_t key;
    if (g >= 0 && g < N) {
      key = t * Npad + (uint32_t)g;
    } else {
      key = kinv;
      err = 1;
    }
    keys[o] = key;
    vals[o] = (uint32_t)o;
    __builtin_nontemporal_store((int32_t)b, bag_of + o);
    if (counts0) atomicAdd(&h0[key & (uint32_t)(nb0 - 1)], 1u);
  }
  if (err) atomicOr(&ctr[C_ERR], ERR_INDEX);
  if (counts0) {  // this tile's counts of the first pass, laid out as the histogram kernel's
    __syncthreads();
    for (int d = threadIdx.x; d < nb0; d += SORT_THREADS) counts0[d * ntiles + tile] = h0[d];
  }
}

__global__ void k_check_offsets(const int64_t* __restrict__ offsets, int64_t NB, int64_t M, int32_t* ctr) {
  int64_t b = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int bad = 0;
  for (; b < NB; b += stride) {
    int64_t lo = offsets[b], hi = offsets[b + 1];
    if (lo < 0 || hi < lo || hi > M) bad = 1;
    if (b == 0 && lo != 0) bad = 1;
    if (b == NB - 1 && hi != M) bad = 1;
  }
  if (bad) atomicOr(&ctr[C_ERR], ERR_OFFSETS);
}

// ---------------------------------------------------------------------------
// LSD radix sort of (key, position), stable, BITS-bit digits (8..11)
// ---------------------------------------------------------------------------
template <int BITS>
__global__ void __launch_bounds__(SORT_THREADS) k_radix_hist(const uint32_t* __restrict__ keys, int n, int shift,
                                                             uint32_t* __restrict__ counts, int ntiles) {
  constexpr int NB = 1 << BITS;
  __shared__ uint32_t h[4][NB];  // one histogram per wave
  // tiles in order, an eighth per XCD: the counts of 32 neighbouring tiles share a
  // cache line, written from one L2, and the scatter reads its tiles' keys again
  // on the same XCD
  const int tile = (int)xcd_block(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int w = threadIdx.x >> 6;
  for (int k = threadIdx.x; k < 4 * NB; k += SORT_THREADS) (&h[0][0])[k] = 0;
  __syncthreads();
  const int base = tile * SORT_TILE;
  if (base + SORT_TILE <= n) {
    // a full tile: the order of the counts does not matter, so 16-byte loads
    const uint4* k4 = reinterpret_cast<const uint4*>(keys + base) + threadIdx.x;
    uint4 v[SORT_ITEMS / 4];
#pragma unroll
    for (int j = 0; j < SORT_ITEMS / 4; ++j) v[j] = k4[j * SORT_THREADS];
#pragma unroll
    for (int j = 0; j < SORT_ITEMS / 4; ++j) {
      atomicAdd(&h[w][(v[j].x >> shift) & (NB - 1)], 1u);
      atomicAdd(&h[w][(v[j].y >> shift) & (NB - 1)], 1u);
      atomicAdd(&h[w][(v[j].z >> shift) & (NB - 1)], 1u);
      atomicAdd(&h[w][(v[j].w >> shift) & (NB - 1)], 1u);
    }
  } else {
    uint32_t k[SORT_ITEMS];
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j) {
      const int i = base + j * SORT_THREADS + threadIdx.x;
      k[j] = i < n ? keys[i] : 0u;
    }
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j)
      if (base + j * SORT_THREADS + (int)threadIdx.x < n) atomicAdd(&h[w][(k[j] >> shift) & (NB - 1)], 1u);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < NB; d += SORT_THREADS)
    counts[d * ntiles + tile] = h[0][d] + h[1][d] + h[2][d] + h[3][d];
}

// one block per digit: exclusive offsets of every tile within that digit, and
// the digit's total (the digit bases are formed by the scatter blocks)
__global__ void __launch_bounds__(256) k_radix_scan(uint32_t* __restrict__ counts, int ntiles,
                                                    uint32_t* __restrict__ totals) {
  __shared__ uint32_t smem[4];
  const int d = blockIdx.x;
  uint32_t running = 0;
  uint32_t* row = counts + (int64_t)d * ntiles;
  for (int start = 0; start < ntiles; start += 256 * 4) {
    uint32_t v[4];
    uint32_t sum = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      int i = start + threadIdx.x * 4 + k;
      v[k] = i < ntiles ? row[i] : 0u;
      sum += v[k];
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan<uint32_t, 256>(sum, smem, &tot);
    uint32_t acc = running + ex;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      int i = start + threadIdx.x * 4 + k;
      if (i < ntiles) row[i] = acc;
      acc += v[k];
    }
    running += tot;
  }
  if (threadIdx.x == 0) totals[d] = running;
}

// Stable scatter.  Wave w of the block owns keys [tile + w*1024, +1024); item j
// of lane l is element w*1024 + j*64 + l, so (w, j, l) order is input order.
// Ranks come from per-wave ballots; the tile is first placed in LDS in digit
// order, then written out so that consecutive threads of one digit write
// consecutive addresses.
template <int BITS>
__global__ void __launch_bounds__(SORT_THREADS) k_radix_scatter(const uint32_t* __restrict__ kin,
                                                                const uint32_t* __restrict__ vin,
                                                                uint32_t* __restrict__ kout,
                                                                uint32_t* __restrict__ vout, int n, int shift,
                                                                const uint32_t* __restrict__ offs, int ntiles,
                                                                const uint32_t* __restrict__ totals) {
  constexpr int NB = 1 << BITS;
  __shared__ uint32_t wh[4][NB];  // per-wave digit counts, then the wave's local base per digit
  __shared__ uint32_t dpos[NB];   // output position of the tile's first key of each digit, less
                                  // that key's position in the tile's digit order
  __shared__ uint32_t sk[SORT_TILE], sv[SORT_TILE];
  __shared__ uint32_t scan_tmp[SORT_THREADS / 64];
  // tiles in order, an eighth per XCD (as in the histogram of the same pass)
  const int tile = (int)xcd_block(blockIdx.x, gridDim.x);
  if (tile >= ntiles) return;
  const int w = threadIdx.x >> 6;
  const int lane = lane_id();
  for (int k = threadIdx.x; k < 4 * NB; k += SORT_THREADS) (&wh[0][0])[k] = 0;
  __syncthreads();
  const int tile0 = tile * SORT_TILE;
  const int base = tile0 + w * (SORT_ITEMS * 64);
  const int nt = n - tile0 < SORT_TILE ? n - tile0 : SORT_TILE;  // keys in this tile
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  uint32_t key[SORT_ITEMS], val[SORT_ITEMS], rk[SORT_ITEMS];
#pragma unroll
  for (int j = 0; j < SORT_ITEMS; ++j) {
    const int i = base + j * 64 + lane;
    const bool ok = i < n;
    key[j] = ok ? kin[i] : 0u;
    val[j] = ok ? vin[i] : 0u;
  }
  // this tile's offset within each digit and the pass's digit totals, loaded with the
  // keys so that the write-out below needs no global read
  constexpr int DPT = (NB + SORT_THREADS - 1) / SORT_THREADS;  // digits per thread
  uint32_t toff[DPT], gt[DPT];
#pragma unroll
  for (int q = 0; q < DPT; ++q) {
    const int d = threadIdx.x * DPT + q;
    toff[q] = d < NB ? offs[d * ntiles + tile] : 0u;
    gt[q] = d < NB ? totals[d] : 0u;
  }
#pragma unroll
  for (int j = 0; j < SORT_ITEMS; ++j) {
    const int i = base + j * 64 + lane;
    const bool ok = i < n;
    const uint32_t dg = (key[j] >> shift) & (NB - 1);
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int b = 0; b < BITS; ++b) {
      const uint64_t m = __ballot((dg >> b) & 1);
      peers &= ((dg >> b) & 1) ? m : ~m;
    }
    const uint32_t before = __popcll(peers & lt);
    const uint32_t cnt = __popcll(peers);
    const uint32_t prev = ok ? wh[w][dg] : 0u;
    rk[j] = prev + before;
    if (ok && before == 0) wh[w][dg] = prev + cnt;
  }
  __syncthreads();
  // tile-local digit starts (exclusive scan over digits of the per-digit totals)
  uint32_t tot[DPT], my = 0;
#pragma unroll
  for (int q = 0; q < DPT; ++q) {
    const int d = threadIdx.x * DPT + q;
    tot[q] = d < NB ? wh[0][d] + wh[1][d] + wh[2][d] + wh[3][d] : 0u;
    my += tot[q];
  }
  uint32_t all;
  uint32_t run = block_excl_scan<uint32_t, SORT_THREADS>(my, scan_tmp, &all);
  // digit bases: exclusive scan of the digit totals of the whole pass
  uint32_t gmy = 0;
#pragma unroll
  for (int q = 0; q < DPT; ++q) gmy += gt[q];
  uint32_t gall;
  uint32_t grun = block_excl_scan<uint32_t, SORT_THREADS>(gmy, scan_tmp, &gall);
#pragma unroll
  for (int q = 0; q < DPT; ++q) {
    const int d = threadIdx.x * DPT + q;
    if (d < NB) {
      dpos[d] = grun + toff[q] - run;
      const uint32_t c0 = wh[0][d], c1 = wh[1][d], c2 = wh[2][d];
      wh[0][d] = run;
      wh[1][d] = run + c0;
      wh[2][d] = run + c0 + c1;
      wh[3][d] = run + c0 + c1 + c2;
    }
    run += tot[q];
    grun += gt[q];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < SORT_ITEMS; ++j) {
    const int i = base + j * 64 + lane;
    if (i < n) {
      const uint32_t dg = (key[j] >> shift) & (NB - 1);
      const uint32_t p = wh[w][dg] + rk[j];
      sk[p] = key[j];
      sv[p] = val[j];
    }
  }
  __syncthreads();
  for (int p = threadIdx.x; p < nt; p += SORT_THREADS) {
    const uint32_t k = sk[p];
    const uint32_t pos = dpos[(k >> shift) & (NB - 1)] + (uint32_t)p;
    kout[pos] = k;
    vout[pos] = sv[p];
  }
}

// A sort of at most one tile: every pass in one workgroup, the keys kept in
// registers and LDS between passes.  Each pass ranks exactly as k_radix_scatter
// does (wave ballots, per-wave digit counts, tile-local digit starts) and places
// the tile in LDS in digit order, which for a single tile is the sorted order of
// that pass.  Reads keys/vals and writes kout/vout (which may be the same arrays).
template <int BITS>
__global__ void __launch_bounds__(SORT_THREADS) k_sort_tile(const uint32_t* kin,
                                                            const uint32_t* vin, uint32_t* kout,
                                                            uint32_t* vout, int n, int npasses, int dbits) {
  constexpr int NB = 1 << BITS;
  __shared__ uint32_t wh[4][NB];  // per-wave digit counts, then the wave's base per digit
  __shared__ uint32_t sk[SORT_TILE], sv[SORT_TILE];
  __shared__ uint32_t scan_tmp[SORT_THREADS / 64];
  const int w = threadIdx.x >> 6;
  const int lane = lane_id();
  const int base = w * (SORT_ITEMS * 64);
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  uint32_t key[SORT_ITEMS], val[SORT_ITEMS], rk[SORT_ITEMS];
#pragma unroll
  for (int j = 0; j < SORT_ITEMS; ++j) {
    const int i = base + j * 64 + lane;
    const bool ok = i < n;
    key[j] = ok ? kin[i] : 0u;
    val[j] = ok ? vin[i] : 0u;
  }
  for (int p = 0; p < npasses; ++p) {
    const int shift = p * dbits;
    for (int k = threadIdx.x; k < 4 * NB; k += SORT_THREADS) (&wh[0][0])[k] = 0;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j) {
      const int i = base + j * 64 + lane;
      const bool ok = i < n;
      const uint32_t dg = (key[j] >> shift) & (NB - 1);
      uint64_t peers = __ballot(ok);
#pragma unroll
      for (int b = 0; b < BITS; ++b) {
        const uint64_t m = __ballot((dg >> b) & 1);
        peers &= ((dg >> b) & 1) ? m : ~m;
      }
      const uint32_t before = __popcll(peers & lt);
      const uint32_t cnt = __popcll(peers);
      const uint32_t prev = ok ? wh[w][dg] : 0u;
      rk[j] = prev + before;
      if (ok && before == 0) wh[w][dg] = prev + cnt;
    }
    __syncthreads();
    constexpr int DPT = (NB + SORT_THREADS - 1) / SORT_THREADS;  // digits per thread
    uint32_t tot[DPT], my = 0;
#pragma unroll
    for (int q = 0; q < DPT; ++q) {
      const int d = threadIdx.x * DPT + q;
      tot[q] = d < NB ? wh[0][d] + wh[1][d] + wh[2][d] + wh[3][d] : 0u;
      my += tot[q];
    }
    uint32_t all;
    uint32_t run = block_excl_scan<uint32_t, SORT_THREADS>(my, scan_tmp, &all);
#pragma unroll
    for (int q = 0; q < DPT; ++q) {
      const int d = threadIdx.x * DPT + q;
      if (d < NB) {
        const uint32_t c0 = wh[0][d], c1 = wh[1][d], c2 = wh[2][d];
        wh[0][d] = run;
        wh[1][d] = run + c0;
        wh[2][d] = run + c0 + c1;
        wh[3][d] = run + c0 + c1 + c2;
      }
      run += tot[q];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j) {
      const int i = base + j * 64 + lane;
      if (i < n) {
        const uint32_t pos = wh[w][(key[j] >> shift) & (NB - 1)] + rk[j];
        sk[pos] = key[j];
        sv[pos] = val[j];
      }
    }
    __syncthreads();
    // element i of the pass's output is the next pass's input element i
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j) {
      const int i = base + j * 64 + lane;
      if (i < n) {
        key[j] = sk[i];
        val[j] = sv[i];
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < SORT_ITEMS; ++j) {
    const int i = base + j * 64 + lane;
    if (i < n) {
      kout[i] = key[j];
      vout[i] = val[j];
    }
  }
}

// ---------------------------------------------------------------------------
// generic scans (tile reduce -> single-block scan of tile sums -> tile scan)
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(SCAN_THREADS) k_scan_reduce(const T* __restrict__ in, int64_t n,
                                                              T* __restrict__ tsum) {
  __shared__ T smem[SCAN_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
  T s = 0;
  for (int j = 0; j < SCAN_ITEMS; ++j) {
    int64_t i = base + j * SCAN_THREADS + threadIdx.x;
    if (i < n) s += in[i];
  }
  T tot;
  block_excl_scan<T, SCAN_THREADS>(s, smem, &tot);
  if (threadIdx.x == 0) tsum[blockIdx.x] = tot;
}

// The sum of v[0 .. count - 1] over the block (every thread gets it): a down-sweep
// block forms its tile's offset from the raw tile totals itself, so no launch scans
// the totals in between (integer sums: the order does not change them).
template <typename T>
__device__ __forceinline__ T block_sum_first(const T* __restrict__ v, int count, T* smem) {
  T s = 0;
  for (int i = threadIdx.x; i < count; i += SCAN_THREADS) s += v[i];
  T tot;
  block_excl_scan<T, SCAN_THREADS>(s, smem, &tot);
  return tot;
}

// each thread scans SCAN_ITEMS consecutive elements; the tile's offset is the sum of
// the tile totals in tsum before it (tsum NULL: a single tile); the last tile writes
// the total to total_out
template <typename T, bool INCLUSIVE>
__global__ void __launch_bounds__(SCAN_THREADS) k_scan_down(const T* __restrict__ in, T* __restrict__ out, int64_t n,
                                                            const T* __restrict__ tsum, int32_t* total_out) {
  __shared__ T smem[SCAN_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + (int64_t)threadIdx.x * SCAN_ITEMS;
  T v[SCAN_ITEMS];
  T s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    int64_t i = base + k;
    v[k] = i < n ? in[i] : (T)0;
    s += v[k];
  }
  const T before = tsum ? block_sum_first<T>(tsum, (int)blockIdx.x, smem) : (T)0;
  T tot;
  T acc = block_excl_scan<T, SCAN_THREADS>(s, smem, &tot) + before;
  if (total_out && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *total_out = (int32_t)(before + tot);
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    int64_t i = base + k;
    if (INCLUSIVE) acc += v[k];
    if (i < n) out[i] = acc;
    if (!INCLUSIVE) acc += v[k];
  }
}

template <typename T, bool INCLUSIVE>
static hipError_t scan_generic(const T* in, T* out, int64_t n, T* tsum, int32_t* total_out, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int ntiles = (int)((n + SCAN_TILE - 1) / SCAN_TILE);
  if (ntiles == 1) {  // one launch
    hipLaunchKernelGGL((k_scan_down<T, INCLUSIVE>), dim3(1), dim3(SCAN_THREADS), 0, st, in, out, n, (const T*)nullptr,
                       total_out);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_scan_reduce<T>, dim3(ntiles), dim3(SCAN_THREADS), 0, st, in, n, tsum);
  hipLaunchKernelGGL((k_scan_down<T, INCLUSIVE>), dim3(ntiles), dim3(SCAN_THREADS), 0, st, in, out, n,
                     (const T*)tsum, total_out);
  return hipGetLastError();
}

hipError_t scan_u32_exclusive(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* tsum, int32_t* total_out,
                              hipStream_t st) {
  return scan_generic<uint32_t, false>(in, out, n, tsum, total_out, st);
}

// ---------------------------------------------------------------------------
// unique rows and prefix groups
// ---------------------------------------------------------------------------
// Unique rows and prefix groups in two passes over the sorted keys.  An
// occurrence starts a row when its key differs from the previous one, and a
// prefix group when, in addition, key / n3 (table and prefix) differs.  Counts
// are packed (rows | groups << 32).
__global__ void __launch_bounds__(SCAN_THREADS) k_group_reduce(const uint32_t* __restrict__ sk, int n, uint32_t kinv,
                                                               uint32_t n3, int dedup, uint64_t* __restrict__ tsum,
                                                               int32_t* __restrict__ ctr) {
  __shared__ uint64_t smem[SCAN_THREADS / 64];
  // each thread counts SCAN_ITEMS consecutive keys (16-byte loads), so a key's
  // predecessor is in a register, and each key's prefix is divided out once
  const int e0 = blockIdx.x * SCAN_TILE + (int)threadIdx.x * SCAN_ITEMS;
  uint32_t k[SCAN_ITEMS];
  if (e0 + SCAN_ITEMS <= n) {
    const uint4* k4 = reinterpret_cast<const uint4*>(sk + e0);
#pragma unroll
    for (int q = 0; q < SCAN_ITEMS / 4; ++q) {
      const uint4 v = k4[q];
      k[4 * q] = v.x;
      k[4 * q + 1] = v.y;
      k[4 * q + 2] = v.z;
      k[4 * q + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int q = 0; q < SCAN_ITEMS; ++q) k[q] = e0 + q < n ? sk[e0 + q] : kinv;
  }
  const uint32_t kprev = e0 > 0 && e0 <= n ? sk[e0 - 1] : 0u;
  const uint32_t knext = e0 + SCAN_ITEMS < n ? sk[e0 + SCAN_ITEMS] : kinv;
  uint64_t c = 0;
  uint32_t pprev = kprev / n3;
#pragma unroll
  for (int q = 0; q < SCAN_ITEMS; ++q) {
    const int i = e0 + q;
    const uint32_t key = k[q], kp = q ? k[q - 1] : kprev;
    const uint32_t pk = key / n3;
    if (i < n && key < kinv) {
      const bool head = i == 0 || kp != key || !dedup;
      const bool pgh = head && (i == 0 || pprev != pk);
      c += (uint64_t)head | ((uint64_t)pgh << 32);
      const uint32_t kn = q + 1 < SCAN_ITEMS ? k[q + 1] : knext;
      if (i == n - 1 || kn >= kinv) ctr[C_NVALID] = i + 1;
    }
    pprev = pk;
  }
  uint64_t tot;
  block_excl_scan<uint64_t, SCAN_THREADS>(c, smem, &tot);
  if (threadIdx.x == 0) tsum[blockIdx.x] = tot;
}

// The tile's keys and positions go through LDS so that each thread scans
// SCAN_ITEMS consecutive occurrences while global reads and writes stay
// coalesced; writes the inverse map, row id per sorted occurrence, unique keys,
// i3 per row, occurrence starts, prefix-group starts and keys.
__device__ __forceinline__ int pad32(int x) { return x + (x >> 5); }

__global__ void __launch_bounds__(SCAN_THREADS) k_group_down(const uint32_t* __restrict__ sk,
                                                             const uint32_t* __restrict__ sp, int n, uint32_t kinv,
                                                             uint32_t n3, uint32_t Npad, int dedup,
                                                             const uint64_t* __restrict__ tsum,
                                                             int32_t* __restrict__ inv, int32_t* __restrict__ sorted_uid,
                                                             uint32_t* __restrict__ uniq_key,
                                                             int32_t* __restrict__ uniq_i3,
                                                             int32_t* __restrict__ occ_start,
                                                             int32_t* __restrict__ pg_start,
                                                             uint32_t* __restrict__ pg_key, int32_t* __restrict__ ctr) {
  // LDS index x is stored at x + x / 32 so that the per-thread runs of
  // SCAN_ITEMS consecutive entries do not all fall on two banks
  __shared__ uint32_t lk[SCAN_TILE + 2 + SCAN_TILE / 32];  // lk[e + 1] = key of tile element e, lk[0] = key before
  __shared__ int32_t lu[SCAN_TILE + SCAN_TILE / 32];        // row id of each element (-1: invalid)
  __shared__ int32_t lg[SCAN_TILE + SCAN_TILE / 32];        // (group id << 1) | group starts here; -1: invalid
  __shared__ uint64_t smem[SCAN_THREADS / 64];
  // tiles in sorted order, an eighth per XCD: a table's inverse-map entries (a
  // contiguous range of positions) are scattered within one XCD's L2, and the
  // kernel's sequential reads and writes are non-temporal so that they do not push
  // those lines out
  const int tile = (int)xcd_block(blockIdx.x, gridDim.x);
  if (tile >= (n + SCAN_TILE - 1) / SCAN_TILE) return;
  const int base = tile * SCAN_TILE;
  // the positions of the thread's striped elements, loaded with the keys so that the
  // inverse-map stores below wait on no load
  uint32_t pos[SCAN_ITEMS];
#pragma unroll
  for (int j = 0; j < SCAN_ITEMS; ++j) {
    const int e = j * SCAN_THREADS + (int)threadIdx.x;
    pos[j] = base + e < n ? __builtin_nontemporal_load(sp + base + e) : 0u;
  }
#pragma unroll 4
  for (int j = 0; j < SCAN_ITEMS; ++j) {
    const int e = j * SCAN_THREADS + (int)threadIdx.x;
    lk[pad32(e + 1)] = base + e < n ? __builtin_nontemporal_load(sk + base + e) : kinv;
  }
  if (threadIdx.x == 0) lk[0] = base > 0 ? sk[base - 1] : 0u;
  __syncthreads();
  // run ids: each thread scans SCAN_ITEMS consecutive elements
  const int e0 = (int)threadIdx.x * SCAN_ITEMS;
  uint32_t hb = 0, pb = 0;  // head / group-head bits of the thread's elements
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int i = base + e0 + k;
    const uint32_t key = lk[pad32(e0 + k + 1)], kp = lk[pad32(e0 + k)];
    if (i < n && key < kinv) {
      const bool head = i == 0 || kp != key || !dedup;
      const bool pgh = head && (i == 0 || kp / n3 != key / n3);
      hb |= (uint32_t)head << k;
      pb |= (uint32_t)pgh << k;
    }
  }
  uint64_t tot;
  const uint64_t c = (uint64_t)__popc(hb) | ((uint64_t)__popc(pb) << 32);
  const uint64_t before = tsum ? block_sum_first<uint64_t>(tsum, tile, smem) : 0ull;
  uint64_t acc = block_excl_scan<uint64_t, SCAN_THREADS>(c, smem, &tot) + before;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int i = base + e0 + k;
    const uint32_t key = lk[pad32(e0 + k + 1)];
    acc += (uint64_t)((hb >> k) & 1) | ((uint64_t)((pb >> k) & 1) << 32);
    const bool valid = i < n && key < kinv;
    lu[pad32(e0 + k)] = valid ? (int)(acc & 0xffffffffu) - 1 : -1;
    lg[pad32(e0 + k)] = valid ? (((int)(acc >> 32) - 1) << 1) | (int)((pb >> k) & 1) : -1;
  }
  __syncthreads();
  // all global writes in striped order (consecutive lanes, consecutive elements)
#pragma unroll
  for (int j = 0; j < SCAN_ITEMS; ++j) {
    const int e = j * SCAN_THREADS + (int)threadIdx.x;
    const int i = base + e;
    if (i >= n) continue;
    const int32_t uid = lu[pad32(e)];
    inv[pos[j]] = uid;
    if (uid < 0) continue;
    __builtin_nontemporal_store(uid, sorted_uid + i);
    const uint32_t key = lk[pad32(e + 1)], kp = lk[pad32(e)];
    if (i == 0 || kp != key || !dedup) {
      __builtin_nontemporal_store(key, uniq_key + uid);
      __builtin_nontemporal_store((int)((key % Npad) % n3), uniq_i3 + uid);
      __builtin_nontemporal_store(i, occ_start + uid);
    }
    const int32_t gv = lg[pad32(e)];
    const int32_t pg = gv >> 1;
    if (gv & 1) {
      pg_start[pg] = uid;
      pg_key[pg] = key / n3;
    }
    const uint32_t knext = e + 1 < SCAN_TILE ? lk[pad32(e + 2)] : (i + 1 < n ? sk[i + 1] : kinv);
    if (i == n - 1 || knext >= kinv) {
      // the last valid occurrence: totals and end sentinels
      ctr[C_NVALID] = i + 1;
      ctr[C_U] = uid + 1;
      ctr[C_P] = pg + 1;
      occ_start[uid + 1] = i + 1;
      pg_start[pg + 1] = uid + 1;
    }
  }
}

// prefix slots in (table, i2, i1) order: slices per group
__global__ void k_dense_set(const int32_t* __restrict__ pg_start, const uint32_t* __restrict__ pg_key,
                            const int32_t* __restrict__ ctr, int n1, int n2, int slice_rows,
                            uint32_t* __restrict__ dense_cnt, int32_t* __restrict__ dense_pg) {
  const int P = ctr[C_P];
  const int n12 = n1 * n2;
  for (int p = blockIdx.x * blockDim.x + threadIdx.x; p < P; p += gridDim.x * blockDim.x) {
    uint32_t key = pg_key[p];
    uint32_t t = key / n12, q = key % n12;
    uint32_t i1 = q / n2, i2 = q % n2;
    int64_t slot = ((int64_t)t * n2 + i2) * n1 + i1;
    int rows = pg_start[p + 1] - pg_start[p];
    dense_cnt[slot] = (uint32_t)((rows + slice_rows - 1) / slice_rows);
    dense_pg[slot] = p;
  }
}

__global__ void k_make_slices(const uint32_t* __restrict__ dense_cnt, const uint32_t* __restrict__ dense_base,
                              const int32_t* __restrict__ dense_pg, int64_t ndense,
                              const int32_t* __restrict__ pg_start, const uint32_t* __restrict__ pg_key, int n1,
                              int slice_rows, int4* __restrict__ slices, int32_t* __restrict__ slice_i1) {
  for (int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; s < ndense;
       s += (int64_t)gridDim.x * blockDim.x) {
    uint32_t c = dense_cnt[s];
    if (!c) continue;
    int p = dense_pg[s];
    uint32_t b = dense_base[s];
    int r0 = pg_start[p], r1 = pg_start[p + 1];
    for (uint32_t k = 0; k < c; ++k) {
      int rb = r0 + (int)k * slice_rows;
      int re = rb + slice_rows < r1 ? rb + slice_rows : r1;
      slices[b + k] = make_int4(p, rb, re, (int)pg_key[p]);
      slice_i1[b + k] = (int)(s % n1);  // slot = (t * n2 + i2) * n1 + i1
    }
  }
}

// One-row slices (reuse ablation levels): one thread per slice, so a hot prefix
// with many occurrences is not written out by a single thread. The slice's slot
// is found by binary search over the exclusive scan of the slice counts.
__global__ void k_make_slices_rows(const uint32_t* __restrict__ dense_base,
                                   const int32_t* __restrict__ dense_pg, int64_t ndense,
                                   const int32_t* __restrict__ pg_start, const uint32_t* __restrict__ pg_key,
                                   int n1, const int32_t* __restrict__ ctr, int4* __restrict__ slices,
                                   int32_t* __restrict__ slice_i1) {
  const int nsl = ctr[C_NSLICES];
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < nsl; x += (int64_t)gridDim.x * blockDim.x) {
    int64_t lo = 0, hi = ndense;  // first slot with base > x, minus one
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (dense_base[mid] <= (uint32_t)x)
        lo = mid + 1;
      else
        hi = mid;
    }
    // An empty slot shares its base with the slot after it, so the last slot whose
    // base does not exceed x is never empty (x < nsl rules out an empty final slot).
    const int64_t slot = lo - 1;
    const int p = dense_pg[slot];
    const int rb = pg_start[p] + (int)((uint32_t)x - dense_base[slot]);
    slices[x] = make_int4(p, rb, rb + 1, (int)pg_key[p]);
    slice_i1[x] = (int)(slot % n1);
  }
}

// chunks of the specialised kernels: up to cs (the shape's chunk_slices) consecutive slices of
// one (t, i2) run; run r covers slices [dense_base[r*n1], dense_base[(r+1)*n1])
__global__ void k_run_counts(const uint32_t* __restrict__ dense_base, const int32_t* __restrict__ ctr, int nruns,
                             int n1, int cs, uint32_t* __restrict__ run_nch) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r > nruns) return;
  if (r == nruns) {  // the scan turns this slot into the total
    run_nch[r] = 0;
    return;
  }
  const uint32_t b0 = dense_base[(int64_t)r * n1];
  const uint32_t b1 = r + 1 < nruns ? dense_base[(int64_t)(r + 1) * n1] : (uint32_t)ctr[C_NSLICES];
  run_nch[r] = (b1 - b0 + cs - 1) / cs;
}

__global__ void k_make_chunks(const uint32_t* __restrict__ dense_base, const uint32_t* __restrict__ run_base,
                              const int32_t* __restrict__ ctr, int nruns, int n1, int cs, int4* __restrict__ chunks) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= nruns) return;
  const uint32_t b0 = dense_base[(int64_t)r * n1];
  const uint32_t b1 = r + 1 < nruns ? dense_base[(int64_t)(r + 1) * n1] : (uint32_t)ctr[C_NSLICES];
  const uint32_t c0 = run_base[r];
  for (uint32_t k = 0; b0 + k * cs < b1; ++k) {
    const uint32_t f = b0 + k * cs;
    const uint32_t n = b1 - f < (uint32_t)cs ? b1 - f : (uint32_t)cs;
    chunks[c0 + k] = make_int4((int)f, (int)n, r, 0);
  }
}

// SCHED_GROUP: chunks are whole prefix groups.  Chunks per prefix slot (a group of
// more than GROUP_CHUNK_MAX slices in pieces), scanned in place into each slot's
// first chunk; a run's first chunk is then that of its first slot.
__global__ void k_slot_chunks(const uint32_t* __restrict__ dense_cnt, int64_t ndense, uint32_t* __restrict__ cnt_out) {
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < ndense; x += (int64_t)gridDim.x * blockDim.x)
    cnt_out[x] = (dense_cnt[x] + GROUP_CHUNK_MAX - 1) / GROUP_CHUNK_MAX;
}
__global__ void k_group_run_base(const uint32_t* __restrict__ slot_base, const int32_t* __restrict__ ctr, int nruns,
                                 int n1, uint32_t* __restrict__ run_base) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < nruns) run_base[r] = slot_base[(int64_t)r * n1];
  if (r == nruns) run_base[r] = (uint32_t)ctr[C_NCHUNKS];
}
__global__ void k_make_group_chunks(const uint32_t* __restrict__ dense_cnt, const uint32_t* __restrict__ dense_base,
                                    const uint32_t* __restrict__ slot_base, int64_t ndense, int n1,
                                    int4* __restrict__ chunks) {
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < ndense; x += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t c = dense_cnt[x];
    for (uint32_t k = 0; k * GROUP_CHUNK_MAX < c; ++k) {
      const uint32_t n = c - k * GROUP_CHUNK_MAX < (uint32_t)GROUP_CHUNK_MAX ? c - k * GROUP_CHUNK_MAX : GROUP_CHUNK_MAX;
      chunks[slot_base[x] + k] = make_int4((int)(dense_base[x] + k * GROUP_CHUNK_MAX), (int)n, (int)(x / n1), 0);
    }
  }
}

// k_run_counts and the scan of its counts in one workgroup when nruns + 1 <=
// SCAN_TILE: chunk counts per run, exclusive scan into run_nch (the total at
// run_nch[nruns] and in ctr[C_NCHUNKS]).  A thread owns SCAN_ITEMS consecutive
// runs.  (The chunk list stays a launch of its own: a run can hold thousands of
// chunks at the no-dedup level.)
__global__ void __launch_bounds__(SCAN_THREADS) k_runs_one_block(const uint32_t* __restrict__ dense_base,
                                                                 int32_t* __restrict__ ctr, int nruns, int n1, int cs,
                                                                 uint32_t* __restrict__ run_nch) {
  __shared__ uint32_t smem[SCAN_THREADS / 64];
  const uint32_t nsl = (uint32_t)ctr[C_NSLICES];
  const int r0 = (int)threadIdx.x * SCAN_ITEMS;
  uint32_t b[SCAN_ITEMS + 1], cnt[SCAN_ITEMS], sum = 0;
#pragma unroll
  for (int k = 0; k <= SCAN_ITEMS; ++k) {
    const int r = r0 + k;
    b[k] = r < nruns ? dense_base[(int64_t)r * n1] : nsl;
  }
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    cnt[k] = r0 + k < nruns ? (b[k + 1] - b[k] + cs - 1) / cs : 0u;
    sum += cnt[k];
  }
  uint32_t tot;
  uint32_t acc = block_excl_scan<uint32_t, SCAN_THREADS>(sum, smem, &tot);
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int r = r0 + k;
    if (r <= nruns) run_nch[r] = acc;
    acc += cnt[k];
  }
  if (threadIdx.x == 0) ctr[C_NCHUNKS] = (int32_t)tot;
}

// Clears what a grouping accumulates into: the counters and the error word, the
// radix digit totals, the dense prefix counts and the tile-to-bag map.
__global__ void k_group_init(int32_t* ctr, int32_t* occ_start, int32_t* pg_start, uint32_t* rtotals,
                             int nrtotals, uint32_t* dense_cnt, int64_t ndense, int32_t* tile_bag, int ntile_bag) {
  const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (i0 < C_TOTAL) ctr[i0] = 0;
  if (i0 < nrtotals) rtotals[i0] = 0;
  if (i0 == 0) {
    occ_start[0] = 0;
    pg_start[0] = 0;
  }
  for (int64_t i = i0; i < ndense; i += stride) dense_cnt[i] = 0u;
  for (int64_t i = i0; i < ntile_bag; i += stride) tile_bag[i] = 0;
}

static int grid_for(int64_t n, int per_block, int cap) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (int)g;
}

// counted: the tile counts of this pass are already in rcounts (the first pass of
// the grouping's sort, counted by the ingest kernel)
template <int BITS>
static hipError_t radix_pass(const Work& w, int cur, int n, int shift, int ntiles, uint32_t* tot, hipStream_t st,
                             bool counted = false) {
  if (!counted)
    hipLaunchKernelGGL(k_radix_hist<BITS>, dim3(xcd_grid(ntiles)), dim3(SORT_THREADS), 0, st, w.keys[cur], n, shift,
                       w.rcounts, ntiles);
  hipLaunchKernelGGL(k_radix_scan, dim3(1 << BITS), dim3(256), 0, st, w.rcounts, ntiles, tot);
  hipLaunchKernelGGL(k_radix_scatter<BITS>, dim3(xcd_grid(ntiles)), dim3(SORT_THREADS), 0, st, w.keys[cur], w.vals[cur],
                     w.keys[cur ^ 1], w.vals[cur ^ 1], n, shift, (const uint32_t*)w.rcounts, ntiles,
                     (const uint32_t*)tot);
  return hipGetLastError();
}

// Stable LSD radix sort of n (key, value) pairs of key_bits-bit keys between the
// ping-pong buffers keys[0..1] / vals[0..1] (input in [0]), with the grouping's
// radix count and total buffers as scratch (the grouping no longer reads them).
// *out receives the buffer index that holds the result.
hipError_t sort_pairs(const Work& w, uint32_t* const keys[2], uint32_t* const vals[2], int n, int key_bits,
                      int* out, hipStream_t st) {
  const int npasses = sort_passes(key_bits < 1 ? 1 : key_bits);
  const int dbits = (key_bits + npasses - 1) / npasses;
  const int bits = dbits < 8 ? 8 : dbits;
  const int ntiles = (n + SORT_TILE - 1) / SORT_TILE;
  Work v = w;
  int cur = 0;
  for (int p = 0; p < npasses && n > 0; ++p) {
    v.keys[0] = keys[0];
    v.keys[1] = keys[1];
    v.vals[0] = vals[0];
    v.vals[1] = vals[1];
    uint32_t* tot = w.rtotals + p * (1 << bits);
    hipError_t e;
    switch (bits) {
      case 8: e = radix_pass<8>(v, cur, n, p * dbits, ntiles, tot, st); break;
      case 9: e = radix_pass<9>(v, cur, n, p * dbits, ntiles, tot, st); break;
      case 10: e = radix_pass<10>(v, cur, n, p * dbits, ntiles, tot, st); break;
      default: e = radix_pass<11>(v, cur, n, p * dbits, ntiles, tot, st); break;
    }
    if (e != hipSuccess) return e;
    cur ^= 1;
  }
  *out = cur;
  return hipGetLastError();
}

hipError_t launch_group(const Shape& s, const Work& w, const int64_t* idx, int64_t M, const int64_t* offsets,
                        int64_t B, const Prof& prof, hipStream_t st) {
  // passes of equal width, at most RADIX_MAX_BITS bits each
  const int npasses = sort_passes(s.key_bits);
  // digit width actually used: 8..11 bits; pass p sorts bits [p dbits, p dbits + bits)
  const int dbits = npasses ? (s.key_bits + npasses - 1) / npasses : 8;
  const int bits = dbits < 8 ? 8 : dbits;
  const int radix = 1 << bits;
  const int nrt = npasses * radix;
  const int64_t NB = (int64_t)s.T * B;
  const int n = M > 0 ? (int)M : 0;
  const int ntiles = (n + SORT_TILE - 1) / SORT_TILE;
  const bool bags = offsets && NB > 0;
  {
    const int ntb = bags && n > 0 ? ntiles + 1 : 0;
    int64_t total = C_TOTAL > nrt ? C_TOTAL : nrt;
    if (s.ndense > total) total = s.ndense;
    if (ntb > total) total = ntb;
    hipLaunchKernelGGL(k_group_init, dim3(grid_for(total, 256, 1024)), dim3(256), 0, st, w.ctr, w.occ_start,
                       w.pg_start, w.rtotals, nrt, w.dense_cnt, (int64_t)s.ndense, w.tile_bag, ntb);
  }
  hipError_t e;
  if (M <= 0) {
    if (bags)
      hipLaunchKernelGGL(k_check_offsets, dim3(grid_for(NB, 256, 1024)), dim3(256), 0, st, offsets, NB, M, w.ctr);
    return hipGetLastError();
  }
  prof_begin(prof, K_INGEST, st);
  if (bags)
    hipLaunchKernelGGL(k_tile_bags, dim3((unsigned)((NB + 255) / 256)), dim3(256), 0, st, offsets, NB, M,
                       w.tile_bag, w.ctr);
  // with more than one tile, ingest also counts the digits of the first sort pass
  const bool count0 = ntiles > 1 && npasses > 0;
  hipLaunchKernelGGL(k_ingest, dim3(xcd_grid(ntiles)), dim3(SORT_THREADS), 0, st, idx, M, offsets, (const int32_t*)w.tile_bag,
                     B, s.T, s.N, s.Npad, s.kinv, w.keys[0], w.vals[0], w.bag_of, w.ctr, count0 ? w.rcounts : nullptr,
                     radix, ntiles);
  prof_end(prof, K_INGEST, st);
  int cur = 0;
  if (ntiles == 1) {
    // one tile: all passes in one launch, the result where the last pass would leave it
    cur = npasses & 1;
    switch (bits) {
      case 8: hipLaunchKernelGGL(k_sort_tile<8>, dim3(1), dim3(SORT_THREADS), 0, st, w.keys[0], w.vals[0],
                                 w.keys[cur], w.vals[cur], n, npasses, dbits); break;
      case 9: hipLaunchKernelGGL(k_sort_tile<9>, dim3(1), dim3(SORT_THREADS), 0, st, w.keys[0], w.vals[0],
                                 w.keys[cur], w.vals[cur], n, npasses, dbits); break;
      case 10: hipLaunchKernelGGL(k_sort_tile<10>, dim3(1), dim3(SORT_THREADS), 0, st, w.keys[0], w.vals[0],
                                  w.keys[cur], w.vals[cur], n, npasses, dbits); break;
      default: hipLaunchKernelGGL(k_sort_tile<11>, dim3(1), dim3(SORT_THREADS), 0, st, w.keys[0], w.vals[0],
                                  w.keys[cur], w.vals[cur], n, npasses, dbits); break;
    }
  } else {
    for (int p = 0; p < npasses; ++p) {
      const int shift = p * dbits;
      uint32_t* tot = w.rtotals + p * radix;
      switch (bits) {
        case 8: e = radix_pass<8>(w, cur, n, shift, ntiles, tot, st, p == 0); break;
        case 9: e = radix_pass<9>(w, cur, n, shift, ntiles, tot, st, p == 0); break;
        case 10: e = radix_pass<10>(w, cur, n, shift, ntiles, tot, st, p == 0); break;
        default: e = radix_pass<11>(w, cur, n, shift, ntiles, tot, st, p == 0); break;
      }
      if (e != hipSuccess) return e;
      cur ^= 1;
    }
  }
  const uint32_t* sk = w.keys[cur];
  const uint32_t* sp = w.vals[cur];
  {
    const int gt = (n + SCAN_TILE - 1) / SCAN_TILE;
    if (gt > 1) {  // a single tile starts at row 0 and group 0: no tile offsets needed
      hipLaunchKernelGGL(k_group_reduce, dim3(gt), dim3(SCAN_THREADS), 0, st, sk, n, s.kinv, (uint32_t)s.n3, s.dedup,
                         w.tsum64, w.ctr);
    }
    hipLaunchKernelGGL(k_group_down, dim3(xcd_grid(gt)), dim3(SCAN_THREADS), 0, st, sk, sp, n, s.kinv, (uint32_t)s.n3, s.Npad,
                       s.dedup, gt > 1 ? (const uint64_t*)w.tsum64 : nullptr, w.inv, w.sorted_uid, w.uniq_key,
                       w.uniq_i3, w.occ_start, w.pg_start, w.pg_key, w.ctr);
  }
  hipLaunchKernelGGL(k_dense_set, dim3(grid_for(M, 256, 2048)), dim3(256), 0, st, (const int32_t*)w.pg_start,
                     (const uint32_t*)w.pg_key, (const int32_t*)w.ctr, s.n1, s.n2, s.slice_rows, w.dense_cnt,
                     w.dense_pg);
  e = scan_generic<uint32_t, false>(w.dense_cnt, w.dense_base, s.ndense, w.tsum32, w.ctr + C_NSLICES, st);
  if (e != hipSuccess) return e;
  if (s.slice_rows == 1)
    hipLaunchKernelGGL(k_make_slices_rows, dim3(grid_for(M, 256, 8192)), dim3(256), 0, st,
                       (const uint32_t*)w.dense_base, (const int32_t*)w.dense_pg,
                       s.ndense, (const int32_t*)w.pg_start, (const uint32_t*)w.pg_key, s.n1, (const int32_t*)w.ctr,
                       w.slices, w.slice_i1);
  else
    hipLaunchKernelGGL(k_make_slices, dim3(grid_for(s.ndense, 256, 4096)), dim3(256), 0, st,
                       (const uint32_t*)w.dense_cnt, (const uint32_t*)w.dense_base, (const int32_t*)w.dense_pg,
                       s.ndense, (const int32_t*)w.pg_start, (const uint32_t*)w.pg_key, s.n1, s.slice_rows,
                       w.slices, w.slice_i1);
  const int nruns = s.T * s.n2;
  if (s.sched == SCHED_GROUP) {
    // slot chunk counts, then their exclusive scan, in dense_pg (free once the slices are made)
    uint32_t* slot_base = reinterpret_cast<uint32_t*>(w.dense_pg);
    hipLaunchKernelGGL(k_slot_chunks, dim3(grid_for(s.ndense, 256, 4096)), dim3(256), 0, st,
                       (const uint32_t*)w.dense_cnt, s.ndense, slot_base);
    e = scan_generic<uint32_t, false>(slot_base, slot_base, s.ndense, w.tsum32, w.ctr + C_NCHUNKS, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_group_run_base, dim3((nruns + 1 + 255) / 256), dim3(256), 0, st, (const uint32_t*)slot_base,
                       (const int32_t*)w.ctr, nruns, s.n1, w.run_nch);
    hipLaunchKernelGGL(k_make_group_chunks, dim3(grid_for(s.ndense, 256, 4096)), dim3(256), 0, st,
                       (const uint32_t*)w.dense_cnt, (const uint32_t*)w.dense_base, (const uint32_t*)slot_base,
                       s.ndense, s.n1, w.chunks);
    return hipGetLastError();
  }
  if (nruns + 1 <= SCAN_TILE) {
    hipLaunchKernelGGL(k_runs_one_block, dim3(1), dim3(SCAN_THREADS), 0, st, (const uint32_t*)w.dense_base, w.ctr,
                       nruns, s.n1, s.chunk_slices, w.run_nch);
  } else {
    hipLaunchKernelGGL(k_run_counts, dim3((nruns + 1 + 255) / 256), dim3(256), 0, st, (const uint32_t*)w.dense_base,
                       (const int32_t*)w.ctr, nruns, s.n1, s.chunk_slices, w.run_nch);
    // exclusive scan in place; the tile sums buffer of the dense scan is free again
    e = scan_generic<uint32_t, false>(w.run_nch, w.run_nch, nruns + 1, w.tsum32, w.ctr + C_NCHUNKS, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_make_chunks, dim3((nruns + 255) / 256), dim3(256), 0, st, (const uint32_t*)w.dense_base,
                     (const uint32_t*)w.run_nch, (const int32_t*)w.ctr, nruns, s.n1, s.chunk_slices, w.chunks);
  return hipGetLastError();
}

}  // namespace ttemb
