// C ABI of libttemb: argument checks, workspace layout and launch order.
// The operator and its conventions are described in include/tt_emb.h.
#include "../../include/tt_emb.h"

#include <mutex>
#include <new>
#include <stdint.h>
#include <string.h>

#include "common.h"

using namespace ttemb;

// Workspace of tt_emb_forward_noalloc: a static array that every GPU the library
// runs on holds until the process ends.  In host code `scratch` only names the
// symbol; its device address comes from hipGetSymbolAddress, once per device
// (scratch_base below), and only that address is passed to kernels.
static __device__ __align__(256) unsigned char scratch[TT_EMB_NOALLOC_SCRATCH_BYTES];

struct tt_emb_s {
  Shape s;
  tt_emb_desc desc;
  // the grouping last written into a workspace, for reuse_grouping = 1
  bool g_valid;
  const void* g_ws;
  const int64_t* g_idx;
  const int64_t* g_off;
  int64_t g_M, g_B;
  Prof prof;  // benchmark event bracketing
};

namespace ttemb {

static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }


// Walks the workspace regions of a call with M indices and B bags per table in
// a fixed order; with base == nullptr it only measures.  Regions that only the
// backward uses come last: *fwd_end receives where they start, so a forward
// call needs fewer bytes than a training step.  The grouping that a forward
// leaves for a backward (reuse_grouping) sits at the same offsets in both, since
// both calls have the same M and B.
static size_t layout(const Shape& s, int64_t M, int64_t B, char* base, Work* w, size_t* fwd_end = nullptr) {
  const int64_t m = M > 0 ? M : 1;
  const int64_t sort_tiles = (m + SORT_TILE - 1) / SORT_TILE;
  const int64_t scan_tiles = (m + SCAN_TILE - 1) / SCAN_TILE;
  const int64_t dscan_tiles = (s.ndense + SCAN_TILE - 1) / SCAN_TILE;
  const int64_t nseg = (m + SEG_CHUNK - 1) / SEG_CHUNK;
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    char* p = base ? base + off : nullptr;
    off = align_up(off + bytes);
    return p;
  };
  Work tmp;
  Work* W = w ? w : &tmp;
  // --- regions of every call: counters, sort, grouping, work list, rows ---
  W->ctr = (int32_t*)take(sizeof(int32_t) * C_TOTAL);
  W->keys[0] = (uint32_t*)take(4 * m);
  W->keys[1] = (uint32_t*)take(4 * m);
  W->vals[0] = (uint32_t*)take(4 * m);
  W->vals[1] = (uint32_t*)take(4 * m);
  W->rcounts = (uint32_t*)take(4 * (size_t)RADIX_MAX * sort_tiles);
  W->tile_bag = (int32_t*)take(4 * (size_t)(sort_tiles + 1));
  W->rtotals = (uint32_t*)take(4 * (size_t)RADIX_MAX * 4);  // at most 3 passes of up to 11 bits
  W->tsum64 = (uint64_t*)take(8 * scan_tiles);
  W->tsum32 = (uint32_t*)take(4 * (dscan_tiles > scan_tiles ? dscan_tiles : scan_tiles));
  W->bag_of = (int32_t*)take(4 * m);
  W->inv = (int32_t*)take(4 * m);
  W->sorted_uid = (int32_t*)take(4 * m);
  W->uniq_key = (uint32_t*)take(4 * m);
  W->uniq_i3 = (int32_t*)take(4 * m);
  W->occ_start = (int32_t*)take(4 * (m + 1));
  W->pg_start = (int32_t*)take(4 * (m + 1));
  W->pg_key = (uint32_t*)take(4 * m);
  W->dense_cnt = (uint32_t*)take(4 * s.ndense);
  W->dense_base = (uint32_t*)take(4 * s.ndense);
  W->dense_pg = (int32_t*)take(4 * s.ndense);
  // Slices: a prefix group of r rows gives ceil(r / slice_rows) < r / slice_rows + 1
  // of them, so there are fewer than U / slice_rows + P <= m / slice_rows + min(ndense, m);
  // with dedup a group also has at most n3 rows, and no slice is empty (at most m).
  const int64_t per_prefix = s.dedup ? (s.n3 + s.slice_rows - 1) / s.slice_rows : m;
  const int64_t groups_max = s.ndense < m ? s.ndense : m;
  int64_t nsl_max = m / s.slice_rows + groups_max + 1;
  if (s.dedup && s.ndense * per_prefix < nsl_max) nsl_max = s.ndense * per_prefix;
  if (nsl_max > m) nsl_max = m;
  // chunks: ceil(slices of run / chunk_slices) per non-empty (t, i2) run, or with
  // SCHED_GROUP ceil(slices of group / GROUP_CHUNK_MAX) per prefix group
  int64_t nch_max = s.sched == SCHED_GROUP ? groups_max + nsl_max / GROUP_CHUNK_MAX + 1
                                           : nsl_max / s.chunk_slices + (int64_t)s.T * s.n2 + 1;
  if (nch_max > nsl_max) nch_max = nsl_max;
  W->nsl_max = nsl_max;
  W->nch_max = nch_max;
  W->slices = (int4*)take(16 * nsl_max);
  W->slice_i1 = (int32_t*)take(4 * nsl_max);
  W->run_nch = (uint32_t*)take(4 * ((int64_t)s.T * s.n2 + 1));
  W->chunks = (int4*)take(16 * nch_max);
  W->E = (float*)take(4 * (size_t)m * s.D);
  // merged first core (L >= 4) or identity middle core (L = 2)
  const size_t nmerged = s.L >= 4 ? (size_t)s.T * s.n1 * s.d1 * s.R : (s.L == 2 ? (size_t)s.T * s.R * s.R : 0);
  W->g1m = nmerged ? (float*)take(4 * nmerged) : nullptr;
  const size_t nlev = (size_t)chain_level_floats(s);
  W->xlev = nlev ? (float*)take(4 * nlev) : nullptr;
  const bool bwd_r32 = bwd_r32_supported(s, m);
  const bool generic = !bwd_r32 || !fwd_r32_supported(s, m);
  const size_t nC = (size_t)s.d1 * s.d2 * s.R;
  W->ckpt = generic ? (float*)take(4 * CKPT_SLOTS * nC) : nullptr;
  W->ckpt_tag = generic ? (int32_t*)take(4 * CKPT_SLOTS) : nullptr;
  if (fwd_end) *fwd_end = off;
  // --- regions of the backward only ---
  W->seg_part = (float*)take(4 * (size_t)nseg * 2 * s.D);
  W->sorted_bag = (int32_t*)take(4 * m);
  // gradient partials: the MFMA backward's rank halves, or the generic backward's
  // per-slice dA, per-chunk dB and per-row dD with the (t, i3) order of the rows
  W->dApart = (float*)take(4 * (size_t)(bwd_r32 ? 2 : 1) * nsl_max * s.d1 * s.R);
  // the R = 64 MFMA backward keeps each slice's dC sum instead of a dB per chunk
  const bool bwd_r64 = !bwd_r32 && bwd_r64_supported(s, m);
  W->dBpart = bwd_r64 ? nullptr : (float*)take(4 * (size_t)nch_max * s.R * s.d2 * s.R);
  W->dCpart = bwd_r64 ? (float*)take(4 * (size_t)nsl_max * s.d1 * s.d2 * s.R) : nullptr;
  W->g3part = bwd_r32 ? (float*)take(4 * (size_t)MAX_BWD_WG * (s.n3 * s.R * s.d3 / 2)) : nullptr;
  W->dDpart = bwd_r32 ? nullptr : (float*)take(4 * (size_t)m * s.R * s.d3);
  for (int k = 0; k < 2; ++k) {
    W->g3keys[k] = bwd_r32 ? nullptr : (uint32_t*)take(4 * m);
    W->g3vals[k] = bwd_r32 ? nullptr : (uint32_t*)take(4 * m);
  }
  W->g3lo = bwd_r32 ? nullptr : (int32_t*)take(4 * (size_t)s.T * s.n3);
  W->g3hi = bwd_r32 ? nullptr : (int32_t*)take(4 * (size_t)s.T * s.n3);
  W->dg1m = nmerged ? (float*)take(4 * nmerged) : nullptr;
  W->dxlev = nlev ? (float*)take(4 * nlev) : nullptr;
  const size_t nsplit = (size_t)split_partial_floats(s);
  W->splitpart = nsplit ? (float*)take(4 * nsplit) : nullptr;
  const int par = sort_passes(s.key_bits) & 1;
  W->sorted_keys = W->keys[par];
  W->sorted_pos = W->vals[par];
  W->M = M;
  W->B = B;
  return off;
}

size_t workspace_bytes(const Shape& s, int64_t M, int64_t B) { return layout(s, M, B, nullptr, nullptr); }

size_t forward_workspace_bytes(const Shape& s, int64_t M, int64_t B) {
  size_t fwd = 0;
  layout(s, M, B, nullptr, nullptr, &fwd);
  return fwd;
}

void carve(const Shape& s, int64_t M, int64_t B, void* base, Work* w) { layout(s, M, B, (char*)base, w); }

__global__ void k_debug_digits(const uint32_t* __restrict__ uniq_key, int U, uint32_t Npad, int n2, int n3,
                               int which, int32_t* __restrict__ out) {
  int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= U) return;
  Digits d = decode_key(uniq_key[u], Npad, n2, n3);
  out[u] = which == 0 ? d.i1 : (which == 1 ? d.i2 : d.i3);
}

// digit `which` (0: i1, 1: i2, 2: i3) of every unique row into out[U]
hipError_t launch_debug_digits(const Shape& s, const Work& w, int32_t* out, int U, int which, hipStream_t st) {
  if (U <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_debug_digits, dim3((U + 255) / 256), dim3(256), 0, st, (const uint32_t*)w.uniq_key, U, s.Npad,
                     s.n2, s.n3, which, out);
  return hipGetLastError();
}

}  // namespace ttemb

static bool al(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// Rows per work slice at the prefix reuse level: 16 on the R = 64 matrix-core shape,
// whose work units are one quad of slices, so that a hot prefix's quads hold at most 32
// row pairs instead of 64 (the heaviest quads otherwise end the launch alone); else
// SLICE_ROWS.
static int prefix_slice_rows(const Shape& s) {
  return s.R == 64 && s.d1 == 4 && s.d2 == 4 && s.d3 == 8 ? 16 : SLICE_ROWS;
}

static int bit_length(uint64_t x) {
  int b = 0;
  while (x) {
    ++b;
    x >>= 1;
  }
  return b;
}

extern "C" {

const char* tt_emb_status_string(tt_emb_status s) {
  switch (s) {
    case TT_EMB_OK: return "ok";
    case TT_EMB_EINVAL: return "invalid argument";
    case TT_EMB_ENOMEM: return "out of host memory";
    case TT_EMB_EHIP: return "HIP runtime error";
    case TT_EMB_ERANGE: return "index or offsets out of range";
    case TT_EMB_EUNSUPPORTED: return "shape not supported";
    case TT_EMB_ESCRATCH: return "call too large for the static scratch of the allocation-free forward";
  }
  return "unknown status";
}

// Validate the three-factor view `d` of a shape with L cores of factors nk, dk
// and create its handle.
static tt_emb_status create_view(const tt_emb_desc* d, int L, const int32_t* nk, const int32_t* dk,
                                 tt_emb_handle* out) {
  const uint64_t npad = (uint64_t)d->row_factors[0] * d->row_factors[1] * d->row_factors[2];
  if ((uint64_t)d->num_rows > npad) return TT_EMB_EINVAL;
  const uint64_t T = (uint64_t)d->num_tables;
  const uint64_t D = (uint64_t)d->dim_factors[0] * d->dim_factors[1] * d->dim_factors[2];
  if (T * npad >= 0xffffffffull) return TT_EMB_EUNSUPPORTED;
  if (T * d->row_factors[0] * d->row_factors[1] >= (1ull << 28)) return TT_EMB_EUNSUPPORTED;
  if ((uint64_t)d->max_indices >= (1ull << 31)) return TT_EMB_EUNSUPPORTED;
  if (T * (uint64_t)d->max_bags >= (1ull << 31)) return TT_EMB_EUNSUPPORTED;
  if (d->rank > 64 || (uint64_t)d->dim_factors[0] * d->dim_factors[1] * d->rank > 8192 || D > 4096)
    return TT_EMB_EUNSUPPORTED;
  tt_emb_s* h = new (std::nothrow) tt_emb_s();
  if (!h) return TT_EMB_ENOMEM;
  h->desc = *d;
  Shape& s = h->s;
  s.T = d->num_tables;
  s.N = d->num_rows;
  s.n1 = d->row_factors[0];
  s.n2 = d->row_factors[1];
  s.n3 = d->row_factors[2];
  s.d1 = d->dim_factors[0];
  s.d2 = d->dim_factors[1];
  s.d3 = d->dim_factors[2];
  s.R = d->rank;
  s.D = (int)D;
  s.Npad = (uint32_t)npad;
  s.kinv = (uint32_t)(T * npad);
  s.key_bits = bit_length(s.kinv);
  s.n12 = s.n1 * s.n2;
  s.ndense = (int64_t)T * s.n1 * s.n2;
  s.slice_rows = prefix_slice_rows(s);
  s.dedup = 1;
  s.sched = SCHED_STEAL;
  s.chunk_slices = s.R == 64 ? TTEMB_R64_CHUNK : TTEMB_CHUNK;
  s.L = L;
  for (int k = 0; k < MAX_CORES; ++k) {
    s.nk[k] = k < L ? nk[k] : 1;
    s.dk[k] = k < L ? dk[k] : 1;
  }
  h->g_valid = false;
  h->prof.kernel = 0;
  h->prof.begin = nullptr;
  h->prof.end = nullptr;
  *out = h;
  return TT_EMB_OK;
}

tt_emb_status tt_emb_create(const tt_emb_desc* d, tt_emb_handle* out) {
  if (!d || !out) return TT_EMB_EINVAL;
  *out = nullptr;
  if (d->num_tables < 1 || d->num_rows < 1 || d->rank < 1 || d->max_indices < 0 || d->max_bags < 0)
    return TT_EMB_EINVAL;
  for (int k = 0; k < 3; ++k)
    if (d->row_factors[k] < 1 || d->dim_factors[k] < 1) return TT_EMB_EINVAL;
  return create_view(d, 3, d->row_factors, d->dim_factors, out);
}

tt_emb_status tt_emb_create_n(const tt_emb_desc_n* d, tt_emb_handle* out) {
  if (!d || !out) return TT_EMB_EINVAL;
  *out = nullptr;
  const int L = d->num_cores;
  if (L < 2 || L > TT_EMB_MAX_CORES || d->num_tables < 1 || d->num_rows < 1 || d->rank < 1 ||
      d->max_indices < 0 || d->max_bags < 0)
    return TT_EMB_EINVAL;
  uint64_t npad = 1, dprod = 1;
  for (int k = 0; k < L; ++k) {
    if (d->row_factors[k] < 1 || d->dim_factors[k] < 1) return TT_EMB_EINVAL;
    npad *= (uint64_t)d->row_factors[k];
    dprod *= (uint64_t)d->dim_factors[k];
    if (npad >= (1ull << 32) || dprod > 4096) return TT_EMB_EUNSUPPORTED;
  }
  if ((uint64_t)d->num_rows > npad) return TT_EMB_EINVAL;
  tt_emb_desc v;
  v.num_tables = d->num_tables;
  v.num_rows = d->num_rows;
  v.rank = d->rank;
  v.max_indices = d->max_indices;
  v.max_bags = d->max_bags;
  if (L == 2) {
    v.row_factors[0] = d->row_factors[0];
    v.row_factors[1] = 1;
    v.row_factors[2] = d->row_factors[1];
    v.dim_factors[0] = d->dim_factors[0];
    v.dim_factors[1] = 1;
    v.dim_factors[2] = d->dim_factors[1];
  } else {
    int64_t n1 = 1, d1 = 1;
    for (int k = 0; k + 2 < L; ++k) {
      n1 *= d->row_factors[k];
      d1 *= d->dim_factors[k];
    }
    if (n1 >= (1 << 28)) return TT_EMB_EUNSUPPORTED;
    v.row_factors[0] = (int32_t)n1;
    v.row_factors[1] = d->row_factors[L - 2];
    v.row_factors[2] = d->row_factors[L - 1];
    v.dim_factors[0] = (int32_t)d1;
    v.dim_factors[1] = d->dim_factors[L - 2];
    v.dim_factors[2] = d->dim_factors[L - 1];
  }
  return create_view(&v, L, d->row_factors, d->dim_factors, out);
}

tt_emb_status tt_emb_profile(tt_emb_handle h, int kernel, void* ev_begin, void* ev_end) {
  if (!h || kernel < TT_EMB_K_NONE || kernel > TT_EMB_K_SPLIT) return TT_EMB_EINVAL;
  const bool off = kernel == TT_EMB_K_NONE || !ev_begin || !ev_end;
  h->prof.kernel = off ? 0 : kernel;
  h->prof.begin = off ? nullptr : (hipEvent_t)ev_begin;
  h->prof.end = off ? nullptr : (hipEvent_t)ev_end;
  return TT_EMB_OK;
}

tt_emb_status tt_emb_kernel_uses_mfma(tt_emb_handle h, int kernel, int64_t num_indices, int* uses_mfma) {
  if (!h || !uses_mfma || kernel < TT_EMB_K_NONE || kernel > TT_EMB_K_SPLIT) return TT_EMB_EINVAL;
  if (num_indices < 0 || num_indices > h->desc.max_indices) return TT_EMB_EINVAL;
  bool m = false;
  if (kernel == TT_EMB_K_FWD_FUSED) m = fwd_r32_supported(h->s, num_indices) || fwd_r64_supported(h->s, num_indices);
  if (kernel == TT_EMB_K_BWD_FUSED) m = bwd_r32_supported(h->s, num_indices) || bwd_r64_supported(h->s, num_indices);
  *uses_mfma = m ? 1 : 0;
  return TT_EMB_OK;
}

tt_emb_status tt_emb_destroy(tt_emb_handle h) {
  delete h;
  return TT_EMB_OK;
}

tt_emb_status tt_emb_set_reuse(tt_emb_handle h, int level) {
  if (!h || level < TT_EMB_REUSE_PREFIX || level > TT_EMB_REUSE_NONE) return TT_EMB_EINVAL;
  h->s.slice_rows = level == TT_EMB_REUSE_PREFIX ? prefix_slice_rows(h->s) : 1;
  h->s.dedup = level == TT_EMB_REUSE_NONE ? 0 : 1;
  h->g_valid = false;  // a grouping made at another level must not be reused
  return TT_EMB_OK;
}

tt_emb_status tt_emb_set_schedule(tt_emb_handle h, int mode) {
  if (!h || mode < TT_EMB_SCHED_STEAL || mode > TT_EMB_SCHED_GROUP) return TT_EMB_EINVAL;
  // the group mode cuts the work list differently: no grouping is reused across it
  if ((mode == TT_EMB_SCHED_GROUP) != (h->s.sched == SCHED_GROUP)) h->g_valid = false;
  h->s.sched = mode;
  return TT_EMB_OK;
}

tt_emb_status tt_emb_workspace_size(tt_emb_handle h, int64_t num_indices, int64_t num_bags, size_t* bytes) {
  if (!h || !bytes) return TT_EMB_EINVAL;
  if (num_indices < 0 || num_bags < 0 || num_indices > h->desc.max_indices || num_bags > h->desc.max_bags)
    return TT_EMB_EINVAL;
  *bytes = workspace_bytes(h->s, num_indices, num_bags);
  return TT_EMB_OK;
}

// Host checks of a call's batch; `training` selects the workspace size of a
// backward (every region) over that of a grouping or forward call.
static tt_emb_status check_batch(tt_emb_handle h, const int64_t* idx, int64_t M, const int64_t* offsets, int64_t B,
                                 const void* ws, size_t ws_bytes, bool training) {
  if (!h || !ws) return TT_EMB_EINVAL;
  if (M < 0 || B < 0 || M > h->desc.max_indices || B > h->desc.max_bags) return TT_EMB_EINVAL;
  if (M > 0 && !idx) return TT_EMB_EINVAL;
  if (!offsets && M != (int64_t)h->s.T * B) return TT_EMB_EINVAL;
  if (offsets && B == 0 && M != 0) return TT_EMB_EINVAL;
  if (!al(idx, 8) || !al(offsets, 8) || !al(ws, 256)) return TT_EMB_EINVAL;
  const size_t need = training ? workspace_bytes(h->s, M, B) : forward_workspace_bytes(h->s, M, B);
  if (ws_bytes < need) return TT_EMB_EINVAL;
  return TT_EMB_OK;
}

static tt_emb_status hip_status(hipError_t e) { return e == hipSuccess ? TT_EMB_OK : TT_EMB_EHIP; }

static tt_emb_status do_group(tt_emb_handle h, const int64_t* idx, int64_t M, const int64_t* offsets, int64_t B,
                              void* ws, hipStream_t st) {
  Work w;
  carve(h->s, M, B, ws, &w);
  h->g_valid = false;
  hipError_t e = launch_group(h->s, w, idx, M, offsets, B, h->prof, st);
  if (e != hipSuccess) return TT_EMB_EHIP;
  h->g_valid = true;
  h->g_ws = ws;
  h->g_idx = idx;
  h->g_off = offsets;
  h->g_M = M;
  h->g_B = B;
  return TT_EMB_OK;
}

static bool grouping_matches(tt_emb_handle h, const int64_t* idx, int64_t M, const int64_t* offsets, int64_t B,
                             const void* ws) {
  return h->g_valid && h->g_ws == ws && h->g_idx == idx && h->g_off == offsets && h->g_M == M && h->g_B == B;
}

tt_emb_status tt_emb_group(tt_emb_handle h, const int64_t* indices, int64_t num_indices, const int64_t* offsets,
                           int64_t num_bags, void* workspace, size_t ws_bytes, void* stream) {
  tt_emb_status st = check_batch(h, indices, num_indices, offsets, num_bags, workspace, ws_bytes, false);
  if (st != TT_EMB_OK) return st;
  return do_group(h, indices, num_indices, offsets, num_bags, workspace, (hipStream_t)stream);
}

tt_emb_status tt_emb_forward(tt_emb_handle h, const float* G1, const float* G2, const float* G3,
                             const int64_t* indices, int64_t num_indices, const int64_t* offsets, int64_t num_bags,
                             float* out, int reuse_grouping, void* workspace, size_t ws_bytes, void* stream) {
  if (h && h->s.L != 3) return TT_EMB_EINVAL;
  tt_emb_status st = check_batch(h, indices, num_indices, offsets, num_bags, workspace, ws_bytes, false);
  if (st != TT_EMB_OK) return st;
  if (!G1 || !G2 || !G3 || (!out && num_bags > 0)) return TT_EMB_EINVAL;
  if (!al(G1, 16) || !al(G2, 16) || !al(G3, 16) || !al(out, 16)) return TT_EMB_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  if (reuse_grouping) {
    if (!grouping_matches(h, indices, num_indices, offsets, num_bags, workspace)) return TT_EMB_EINVAL;
  } else {
    st = do_group(h, indices, num_indices, offsets, num_bags, workspace, s);
    if (st != TT_EMB_OK) return st;
  }
  Work w;
  carve(h->s, num_indices, num_bags, workspace, &w);
  return hip_status(launch_forward(h->s, w, G1, G2, G3, offsets, num_indices, num_bags, out, h->prof, s));
}

// Device address of `scratch` on the current device, looked up on the first call
// made there and kept per device (each device holds its own copy of the array).
static std::mutex g_scratch_mu;
static void* g_scratch_dev[TT_EMB_NOALLOC_MAX_DEVICES];

static tt_emb_status scratch_base(hipStream_t stream, void** base) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return TT_EMB_EHIP;
  if (dev < 0 || dev >= TT_EMB_NOALLOC_MAX_DEVICES) return TT_EMB_EUNSUPPORTED;
  if (stream) {  // the stream must belong to the current device, whose copy is looked up
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return TT_EMB_EHIP;
    if ((int)sdev != dev) return TT_EMB_EINVAL;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TT_EMB_EHIP;
    g_scratch_dev[dev] = p;
  }
  *base = g_scratch_dev[dev];
  return TT_EMB_OK;
}

tt_emb_status tt_emb_forward_noalloc(tt_emb_handle h, const float* G1, const float* G2, const float* G3,
                                     const int64_t* indices, int64_t num_indices, const int64_t* offsets,
                                     int64_t num_bags, float* out, void* stream) {
  if (!h || h->s.L != 3) return TT_EMB_EINVAL;
  if (num_indices < 0 || num_bags < 0 || num_indices > h->desc.max_indices || num_bags > h->desc.max_bags)
    return TT_EMB_EINVAL;
  if (forward_workspace_bytes(h->s, num_indices, num_bags) > (size_t)TT_EMB_NOALLOC_SCRATCH_BYTES)
    return TT_EMB_ESCRATCH;
  hipStream_t s = (hipStream_t)stream;
  void* base = nullptr;
  tt_emb_status st = scratch_base(s, &base);
  if (st != TT_EMB_OK) return st;
  // the checks of tt_emb_forward, with the scratch as the workspace
  st = check_batch(h, indices, num_indices, offsets, num_bags, base, TT_EMB_NOALLOC_SCRATCH_BYTES, false);
  if (st != TT_EMB_OK) return st;
  if (!G1 || !G2 || !G3 || (!out && num_bags > 0)) return TT_EMB_EINVAL;
  if (!al(G1, 16) || !al(G2, 16) || !al(G3, 16) || !al(out, 16)) return TT_EMB_EINVAL;
  // grouped into the scratch (no grouping of the caller's workspace is touched or
  // recorded); the grouping's launches clear every counter and table they rely on
  Work w;
  carve(h->s, num_indices, num_bags, base, &w);
  if (launch_group(h->s, w, indices, num_indices, offsets, num_bags, h->prof, s) != hipSuccess)
    return TT_EMB_EHIP;
  return hip_status(launch_forward(h->s, w, G1, G2, G3, offsets, num_indices, num_bags, out, h->prof, s));
}

tt_emb_status tt_emb_backward(tt_emb_handle h, const float* G1, const float* G2, const float* G3,
                              const int64_t* indices, int64_t num_indices, const int64_t* offsets,
                              int64_t num_bags, const float* grad_out, float* dG1, float* dG2, float* dG3,
                              int reuse_grouping, void* workspace, size_t ws_bytes, void* stream) {
  if (h && h->s.L != 3) return TT_EMB_EINVAL;
  tt_emb_status st = check_batch(h, indices, num_indices, offsets, num_bags, workspace, ws_bytes, true);
  if (st != TT_EMB_OK) return st;
  if (!G1 || !G2 || !G3 || !dG1 || !dG2 || !dG3 || (!grad_out && num_bags > 0)) return TT_EMB_EINVAL;
  if (!al(G1, 16) || !al(G2, 16) || !al(G3, 16) || !al(grad_out, 16) || !al(dG1, 16) || !al(dG2, 16) ||
      !al(dG3, 16))
    return TT_EMB_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  if (reuse_grouping) {
    if (!grouping_matches(h, indices, num_indices, offsets, num_bags, workspace)) return TT_EMB_EINVAL;
  } else {
    st = do_group(h, indices, num_indices, offsets, num_bags, workspace, s);
    if (st != TT_EMB_OK) return st;
  }
  Work w;
  carve(h->s, num_indices, num_bags, workspace, &w);
  return hip_status(
      launch_backward(h->s, w, G1, G2, G3, offsets, num_indices, num_bags, grad_out, dG1, dG2, dG3, 0.f, false,
                      h->prof, s));
}

tt_emb_status tt_emb_backward_sgd(tt_emb_handle h, float* G1, float* G2, float* G3, const int64_t* indices,
                                  int64_t num_indices, const int64_t* offsets, int64_t num_bags,
                                  const float* grad_out, float lr, int reuse_grouping, void* workspace,
                                  size_t ws_bytes, void* stream) {
  if (h && h->s.L != 3) return TT_EMB_EINVAL;
  tt_emb_status st = check_batch(h, indices, num_indices, offsets, num_bags, workspace, ws_bytes, true);
  if (st != TT_EMB_OK) return st;
  if (!G1 || !G2 || !G3 || (!grad_out && num_bags > 0)) return TT_EMB_EINVAL;
  if (!al(G1, 16) || !al(G2, 16) || !al(G3, 16) || !al(grad_out, 16)) return TT_EMB_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  if (reuse_grouping) {
    if (!grouping_matches(h, indices, num_indices, offsets, num_bags, workspace)) return TT_EMB_EINVAL;
  } else {
    st = do_group(h, indices, num_indices, offsets, num_bags, workspace, s);
    if (st != TT_EMB_OK) return st;
  }
  Work w;
  carve(h->s, num_indices, num_bags, workspace, &w);
  return hip_status(launch_backward(h->s, w, G1, G2, G3, offsets, num_indices, num_bags, grad_out, G1, G2, G3, lr,
                                    true, h->prof, s));
}

tt_emb_status tt_emb_sgd(tt_emb_handle h, float* G1, float* G2, float* G3, const float* dG1, const float* dG2,
                         const float* dG3, float lr, void* stream) {
  if (!h || h->s.L != 3 || !G1 || !G2 || !G3 || !dG1 || !dG2 || !dG3) return TT_EMB_EINVAL;
  if (!al(G1, 16) || !al(G2, 16) || !al(G3, 16) || !al(dG1, 16) || !al(dG2, 16) || !al(dG3, 16))
    return TT_EMB_EINVAL;
  return hip_status(launch_sgd(h->s, G1, G2, G3, dG1, dG2, dG3, lr, (hipStream_t)stream));
}

static bool cores_ok(tt_emb_handle h, const float* const* p) {
  if (!p) return false;
  for (int k = 0; k < h->s.L; ++k)
    if (!p[k] || !al(p[k], 16)) return false;
  return true;
}

static tt_emb_status group_or_reuse(tt_emb_handle h, const int64_t* idx, int64_t M, const int64_t* offsets,
                                    int64_t B, void* ws, int reuse_grouping, hipStream_t s) {
  if (reuse_grouping) return grouping_matches(h, idx, M, offsets, B, ws) ? TT_EMB_OK : TT_EMB_EINVAL;
  return do_group(h, idx, M, offsets, B, ws, s);
}

tt_emb_status tt_emb_forward_n(tt_emb_handle h, const float* const* cores, const int64_t* indices,
                               int64_t num_indices, const int64_t* offsets, int64_t num_bags, float* out,
                               int reuse_grouping, void* workspace, size_t ws_bytes, void* stream) {
  tt_emb_status st = check_batch(h, indices, num_indices, offsets, num_bags, workspace, ws_bytes, false);
  if (st != TT_EMB_OK) return st;
  if (!cores_ok(h, cores) || (!out && num_bags > 0) || !al(out, 16)) return TT_EMB_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  if ((st = group_or_reuse(h, indices, num_indices, offsets, num_bags, workspace, reuse_grouping, s)) != TT_EMB_OK)
    return st;
  Work w;
  carve(h->s, num_indices, num_bags, workspace, &w);
  const int L = h->s.L;
  const float *G1 = cores[0], *G2 = cores[1], *G3 = cores[L - 1];
  hipError_t e = hipSuccess;
  if (L == 2) {
    e = launch_identity(h->s, w, s);
    G2 = w.g1m;
  } else if (L >= 4) {
    e = launch_merge(h->s, w, cores, h->prof, s);
    G1 = w.g1m;
    G2 = cores[L - 2];
  }
  if (e != hipSuccess) return TT_EMB_EHIP;
  return hip_status(launch_forward(h->s, w, G1, G2, G3, offsets, num_indices, num_bags, out, h->prof, s));
}

tt_emb_status tt_emb_backward_n(tt_emb_handle h, const float* const* cores, const int64_t* indices,
                                int64_t num_indices, const int64_t* offsets, int64_t num_bags, const float* grad_out,
                                float* const* grads, int reuse_grouping, void* workspace, size_t ws_bytes,
                                void* stream) {
  tt_emb_status st = check_batch(h, indices, num_indices, offsets, num_bags, workspace, ws_bytes, true);
  if (st != TT_EMB_OK) return st;
  if (!cores_ok(h, cores) || !cores_ok(h, (const float* const*)grads) || (!grad_out && num_bags > 0) ||
      !al(grad_out, 16))
    return TT_EMB_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  if ((st = group_or_reuse(h, indices, num_indices, offsets, num_bags, workspace, reuse_grouping, s)) != TT_EMB_OK)
    return st;
  Work w;
  carve(h->s, num_indices, num_bags, workspace, &w);
  const int L = h->s.L;
  const float *G1 = cores[0], *G2 = cores[1], *G3 = cores[L - 1];
  float *dG1 = grads[0], *dG2 = grads[1], *dG3 = grads[L - 1];
  hipError_t e = hipSuccess;
  if (L == 2) {
    e = launch_identity(h->s, w, s);
    G2 = w.g1m;
    dG2 = w.dg1m;
  } else if (L >= 4) {
    e = launch_merge(h->s, w, cores, h->prof, s);
    G1 = w.g1m;
    G2 = cores[L - 2];
    dG1 = w.dg1m;
    dG2 = grads[L - 2];
  }
  if (e != hipSuccess) return TT_EMB_EHIP;
  e = launch_backward(h->s, w, G1, G2, G3, offsets, num_indices, num_bags, grad_out, dG1, dG2, dG3, 0.f, false,
                      h->prof, s);
  if (e != hipSuccess) return TT_EMB_EHIP;
  if (L >= 4) return hip_status(launch_split(h->s, w, cores, grads, h->prof, s));
  return TT_EMB_OK;
}

tt_emb_status tt_emb_sgd_n(tt_emb_handle h, float* const* cores, const float* const* grads, float lr,
                           void* stream) {
  if (!h || !cores_ok(h, (const float* const*)cores) || !cores_ok(h, grads)) return TT_EMB_EINVAL;
  for (int k = 0; k < h->s.L; ++k) {
    hipError_t e = launch_sgd1(cores[k], grads[k], core_elems(h->s, k), lr, (hipStream_t)stream);
    if (e != hipSuccess) return TT_EMB_EHIP;
  }
  return TT_EMB_OK;
}

tt_emb_status tt_emb_check_errors(tt_emb_handle h, void* workspace, void* stream) {
  if (!h || !workspace) return TT_EMB_EINVAL;
  Work w;
  carve(h->s, 0, 0, workspace, &w);  // the counters head every layout
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return TT_EMB_EHIP;
  int32_t err = 0;
  if (hipMemcpy(&err, w.ctr + C_ERR, sizeof(err), hipMemcpyDeviceToHost) != hipSuccess) return TT_EMB_EHIP;
  if (err) {
    int32_t zero = 0;
    if (hipMemcpy(w.ctr + C_ERR, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess) return TT_EMB_EHIP;
    return TT_EMB_ERANGE;
  }
  return TT_EMB_OK;
}

tt_emb_status tt_emb_debug_grouping(tt_emb_handle h, void* workspace, int64_t* uniq_keys, int32_t* uniq_digits,
                                    int32_t* inv, int32_t* occ_start, int32_t* occ_pos, int32_t* pg_start,
                                    int64_t* pg_keys, int64_t* counts, void* stream) {
  if (!h || !workspace) return TT_EMB_EINVAL;
  if (!h->g_valid || h->g_ws != workspace) return TT_EMB_EINVAL;
  hipStream_t st = (hipStream_t)stream;
  Work w;
  carve(h->s, h->g_M, h->g_B, workspace, &w);  // the layout of the grouped call
  if (hipStreamSynchronize(st) != hipSuccess) return TT_EMB_EHIP;
  int32_t c[8];
  if (hipMemcpy(c, w.ctr, sizeof(c), hipMemcpyDeviceToHost) != hipSuccess) return TT_EMB_EHIP;
  const int U = c[C_U], P = c[C_P], nv = c[C_NVALID];
  if (counts) {
    counts[0] = U;
    counts[1] = P;
    counts[2] = nv;
    counts[3] = c[C_NSLICES];
  }
  const int64_t M = h->g_M;
  bool ok = true;
  if (uniq_keys && U > 0) {
    uint32_t* tmp = new (std::nothrow) uint32_t[U];
    if (!tmp) return TT_EMB_ENOMEM;
    ok &= hipMemcpy(tmp, w.uniq_key, 4 * (size_t)U, hipMemcpyDeviceToHost) == hipSuccess;
    for (int i = 0; i < U; ++i) uniq_keys[i] = tmp[i];
    delete[] tmp;
  }
  if (uniq_digits && U > 0) {
    // decoded on the device by the kernels' own key decoder, one digit at a time,
    // into the radix buffer that the sort no longer needs
    int32_t* scratch = reinterpret_cast<int32_t*>(w.sorted_keys == w.keys[0] ? w.keys[1] : w.keys[0]);
    int32_t* tmp = new (std::nothrow) int32_t[U];
    if (!tmp) return TT_EMB_ENOMEM;
    for (int k = 0; k < 3 && ok; ++k) {
      ok &= launch_debug_digits(h->s, w, scratch, U, k, st) == hipSuccess;
      ok &= hipStreamSynchronize(st) == hipSuccess;
      ok &= hipMemcpy(tmp, scratch, 4 * (size_t)U, hipMemcpyDeviceToHost) == hipSuccess;
      for (int i = 0; i < U; ++i) uniq_digits[3 * i + k] = tmp[i];
    }
    delete[] tmp;
  }
  if (inv && M > 0) ok &= hipMemcpy(inv, w.inv, 4 * (size_t)M, hipMemcpyDeviceToHost) == hipSuccess;
  if (occ_start) ok &= hipMemcpy(occ_start, w.occ_start, 4 * (size_t)(U + 1), hipMemcpyDeviceToHost) == hipSuccess;
  if (occ_pos && nv > 0)
    ok &= hipMemcpy(occ_pos, w.sorted_pos, 4 * (size_t)nv, hipMemcpyDeviceToHost) == hipSuccess;
  if (pg_start) ok &= hipMemcpy(pg_start, w.pg_start, 4 * (size_t)(P + 1), hipMemcpyDeviceToHost) == hipSuccess;
  if (pg_keys && P > 0) {
    uint32_t* tmp = new (std::nothrow) uint32_t[P];
    if (!tmp) return TT_EMB_ENOMEM;
    ok &= hipMemcpy(tmp, w.pg_key, 4 * (size_t)P, hipMemcpyDeviceToHost) == hipSuccess;
    for (int i = 0; i < P; ++i) pg_keys[i] = tmp[i];
    delete[] tmp;
  }
  return ok ? TT_EMB_OK : TT_EMB_EHIP;
}

}  // extern "C"
