// Backward pass for R = 32 and d = (4, 4, 8) (D = 128) or d = (4, 4, 2) (D = 32) on MFMA
// (FlowTT Section 3.2, Eq. 1).
//
// Work is split by table t and by half h of the rank index b of the last
// core (b = 16 h + b'), so each (t, h) owner does its half of every product
// exactly once and keeps its half of dG3[t] (n3 x 16 x 8 floats) in LDS:
//   C_h   = A . B_h                 (4 x 64 per group; B_h = G2[i2][:, :, 16h:16h+16])
//   dD_h  = C_h^T . dE_u            -> LDS accumulator of dG3[t][i3][16h + b'][j3]
//   dC_h  = dE_u . D_{u,h}^T, summed over the group's rows into dC_h
//   dB_h += A^T . dC_h              (32 x 64, summed over the chunk's groups)
//   dA_h  = dC_h . B_h^T            (4 x 32, half of the sum over (j2, b))
// A chunk is up to 32 slices of one (t, i2) run, processed four at a time
// ("quads") so stage 1 and dA use 16-row MFMA tiles.  dB_h of a chunk and
// dA_h of a slice go to scratch; three small kernels finish dG1, dG2 and dG3
// by fixed-order segment sums.  Workgroup blockIdx % (2T) owns (t, h), so
// with T = 8 every table lives on one XCD (blockIdx % 8).
// The per-row products take the rows of a slice in groups of 16 / d3 (pairs for
// d3 = 8, eights for d3 = 2), so that a group's (row, j3) columns fill one MFMA tile.
#include "common.h"

namespace ttemb {

ShapeArgs shape_args(const Shape& s);

constexpr int BW_WAVES = 8;
// Per-wave scratch: the quad's [slice][j1][(j2, b')] stack (16 rows of 64 floats),
// first C_h, then dC_h, with rows SCR_PITCH floats apart.  The 4-float pad makes
// every access a per-lane constant base plus an immediate offset and keeps the
// C writes, C^T reads and dA operand reads at the two-lanes-per-bank minimum
// (the dC writes, four per slice, take four lanes per bank).
constexpr int SCR_PITCH = 68;
constexpr int BW_SCR = 16 * SCR_PITCH;

// The LDS dG3 accumulator holds, per table row i3, 16 d3 floats ordered
// [j3][16 slots]: rank row b' = 4 g + r of column j3 sits at slot
// 4 ((g + (j3 >> 1)) & 3) + r.  A dD tile gives lane (j3, g) the four
// consecutive slots of its column, and the rotation by j3 >> 1 spreads the
// lanes of one 16-byte access over all banks.
__device__ __forceinline__ uint32_t g3_slot_base(int j3, int g) {
  return (uint32_t)(j3 * 16 + 4 * ((g + (j3 >> 1)) & 3));
}
__device__ __forceinline__ int g3_unslot(int j3, int p) {  // slot p of column j3 -> b'
  return 4 * (((p >> 2) - (j3 >> 1)) & 3) + (p & 3);
}

// Adds to LDS floats shared by the workgroup's waves.  A float ds_add is slow on
// this LDS, integer compare-and-swap is not: read two floats as a 64-bit word,
// add, swap, and retry from the returned word if it changed in between
// (lock-free: a failed swap means another wave's add landed).
__device__ __forceinline__ uint64_t add2(uint64_t w, float a, float b) {
  const float lo = __uint_as_float((uint32_t)w) + a, hi = __uint_as_float((uint32_t)(w >> 32)) + b;
  return (uint64_t)__float_as_uint(lo) | ((uint64_t)__float_as_uint(hi) << 32);
}
// Compare-and-swap returning the old word only (equal to cmp exactly when the swap
// took place), so that checking the result can wait until it is needed.
__device__ __forceinline__ uint64_t lds_cas_old(uint64_t* u, uint64_t cmp, uint64_t val) {
  __hip_atomic_compare_exchange_strong(u, &cmp, val, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_WORKGROUP);
  return cmp;
}


// operands of one row group.  d3 = 8: rows r0 and r0 + 1 of a slice (a lone last
// row pairs with a row of zeros, which its buffer loads return past the end of the
// pair), with the layouts below.  d3 = 2: up to eight rows (rows past the last read
// as zeros), with eb the 16 bytes of dE[row l15 / 2][8 l4 .. 8 l4 + 7] this lane loads
// (the first half on even lanes, the second on odd), e4 = dE[rows 2 l4, 2 l4 + 1][2 l15
// .. 2 l15 + 1] and d4 = G3[i3 of those rows][16 h + l15][0 .. 1]
struct BwPair {
  float eb[4];  // dD B operand: dE[row][(4 s + l4) * 8 + j3], row r0 in lanes 0-7 of each 16, r0 + 1 in 8-15
  float4 e4;    // dC A operand: dE[row l4 >> 1][l15 * 8 + 4 (l4 & 1) + k]
  float4 d4;    // dC B operand: G3[i3 of that row][16 h + l15][4 (l4 & 1) + k]
  int i3m;      // accumulator row of this lane's dD column: i3 of its row, or for the
                // zero row's column (exact zeros) a neighbouring i3, so that its no-op
                // swap never targets the same words as a live lane of the pair
  int j;        // the pair's slice within the quad (wave-uniform)
};

template <int D3>
__global__ void __launch_bounds__(64 * BW_WAVES, 1)
    k_bwd_r32(ShapeArgs s, const float* __restrict__ G1, const float* __restrict__ G2, const float* __restrict__ G3,
              const float* __restrict__ dE, const int4* __restrict__ slices, const int32_t* __restrict__ slice_i1,
              const int4* __restrict__ chunks, const uint32_t* __restrict__ run_base,
              const int32_t* __restrict__ uniq_i3, int32_t* __restrict__ ctr, float* __restrict__ dApart,
              float* __restrict__ dBpart, float* __restrict__ g3part, int nsl_cap, int nch_cap) {
  extern __shared__ float lds[];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  constexpr int GR = 16 / D3;     // rows per group
  constexpr int DW = 16 * D3;     // floats per dE row
  constexpr int AROW = 16 * D3;   // floats per accumulator row (half the rank of a G3 row)
  // LDS pitch of an accumulator row: at d3 = 2 rows of 32 floats would put every row on one
  // of two bank offsets, so the eight random rows of a group would meet on the same banks;
  // 36 floats spread them over sixteen
  constexpr int APITCH = D3 == 2 ? 36 : AROW;
  const int acc_n = s.n3 * AROW;
  // d3 = 2: eight more rows after the table's, which the columns of a group's missing
  // rows (exact zeros) go to, one per row position, so they never meet a live column
  const int acc_lds = (s.n3 + (D3 == 2 ? 8 : 0)) * APITCH;
  float* g3acc = lds;  // [n3][j3][16 slots]
  float* scr = lds + acc_lds + wave * BW_SCR;
  const int nq = 2 * s.T;
  const int q = blockIdx.x % nq;
  const int t = q % s.T, h = q / s.T;
  int32_t* qctr = ctr + C_BWD_CTR + q * SCHED_STRIDE;  // the owner's queue: all of table t's chunks

  for (int i = threadIdx.x; i < acc_lds; i += blockDim.x) g3acc[i] = 0.f;
  __syncthreads();

  const int c_lo = (int)run_base[t * s.n2], c_hi = (int)run_base[(t + 1) * s.n2];
  const int nch = c_hi - c_lo;
  const int l15 = lane & 15, l4 = lane >> 4;
  const bool rowsel = (l15 >> 3) != 0;  // d3 = 8: dD column of row r0 + 1
  const bool prow = (l4 >> 1) != 0;     // d3 = 8: dC K slots of row r0 + 1
  const int asel = l15 / D3;            // group row of this lane's dD column
  const bool odd_lane = (lane & 1) != 0;
  // per-lane float offsets; every operand is a uniform base plus one of these
  // byte offsets of this lane's operand words: in a group's dE rows and in a G3[t] row
  const uint32_t vo_eb = D3 == 8 ? 4u * (uint32_t)(l4 * 8 + (lane & 7) + (rowsel ? 128 : 0))
                                 : 4u * (uint32_t)(DW * asel + 8 * l4 + 4 * (lane & 1));
  const uint32_t vo_e4 = D3 == 8 ? 4u * (uint32_t)(l15 * 8 + 4 * (l4 & 1) + (prow ? 128 : 0))
                                 : 4u * (uint32_t)(2 * l4 * DW + 2 * l15);
  const uint32_t vo_d4 = D3 == 8 ? 4u * (uint32_t)((16 * h + l15) * 8 + 4 * (l4 & 1)) : 4u * (uint32_t)((16 * h + l15) * 2);
  const uint32_t o_g3 = g3_slot_base(l15 % D3, l4);  // this lane's four dD values in an accumulator row
  const float* G1t = G1 + (uint32_t)(t * s.n1) * 128u;
  const float* G3t = G3 + (uint32_t)(t * s.n3) * (32u * D3);
  // this lane's scratch bases: C write (row 4 l4 + r, column 16 nt + l15), dC write
  // (row 4 j + l4, column 16 r + l15) and dA operand read (row l15, columns 16 l4 + s)
  float* scr_c = scr + 4 * SCR_PITCH * l4 + l15;
  float* scr_d = scr + SCR_PITCH * l4 + l15;
  const float* scr_a = scr + SCR_PITCH * l15 + 16 * l4;
  const buf_t g3buf = make_buf(G3t, (uint32_t)s.n3 * (128u * D3));

  int cursor = 0;
  int cur_run = -1;
  float Bop[32];   // stage-1 B operand B_h[a = 4 s + l4][16 nt + l15], (s, nt) -> 4 s + nt
  float BTop[32];  // dA B operand B_h^T[(j2 = l4, b' = s)][a = 16 nt2 + l15], (s, nt2) -> 16 nt2 + s
  f32x4 dB[8];     // (mt, nt) -> 4 mt + nt; zeroed here and after each chunk's partial is stored
#pragma unroll
  for (int k = 0; k < 8; ++k) dB[k] = f32x4{0.f, 0.f, 0.f, 0.f};

  // slice descriptors of the current chunk, lane j holding slice f + j (j < ns;
  // other lanes have no rows): first row, row count, i1
  int c_rb = 0, c_nr = 0, c_i1 = 0;
  int qd = 0;  // first slice of the current quad within the chunk
  // Row-group descriptors of a quad, lane P holding group P (P < np; slice j owns
  // ceil(nr_j / GR) consecutive groups): the group's first row, and packed, for
  // d3 = 8 i3 of its two rows (8 bits each, n3 <= 256), its slice j and whether the
  // second row is real; for d3 = 2 the position of its first row in the quad's row
  // list (slice 0's rows, then slice 1's, ...: at most 128), its slice j and its row
  // count - 1, with the list's i3 values in lanes L and L + 64 of d_i3lo / d_i3hi.
  // Built one quad ahead (e_*) so the i3 loads are in flight meanwhile.
  int d_ra = 0, d_pk = 0, np = 0;
  int e_ra = 0, e_ia = 0, e_ib = 0, e_jh = 0, e_np = 0;
  int d_i3lo = 0, d_i3hi = 0, e_i3lo = 0, e_i3hi = 0;
  auto build_desc = [&](int qd0) {
    const int n0 = __builtin_amdgcn_readlane(c_nr, qd0), n1 = __builtin_amdgcn_readlane(c_nr, qd0 + 1);
    const int n2 = __builtin_amdgcn_readlane(c_nr, qd0 + 2), n3 = __builtin_amdgcn_readlane(c_nr, qd0 + 3);
    const int b0 = __builtin_amdgcn_readlane(c_rb, qd0), b1 = __builtin_amdgcn_readlane(c_rb, qd0 + 1);
    const int b2 = __builtin_amdgcn_readlane(c_rb, qd0 + 2), b3 = __builtin_amdgcn_readlane(c_rb, qd0 + 3);
    const int q1 = (n0 + GR - 1) / GR, q2 = q1 + (n1 + GR - 1) / GR, q3 = q2 + (n2 + GR - 1) / GR;
    e_np = q3 + (n3 + GR - 1) / GR;
    // group P of slice j starts at row base_j + GR P and holds min(GR, lim_j - GR P)
    // rows, with the wave-uniform base_j = b_j - GR q_j, lim_j = n_j + GR q_j
    const bool s1 = lane >= q1, s2 = lane >= q2, s3 = lane >= q3;
    const int j = (int)s1 + (int)s2 + (int)s3;
    int base = b0, lim = n0;
    base = s1 ? b1 - GR * q1 : base;
    lim = s1 ? n1 + GR * q1 : lim;
    base = s2 ? b2 - GR * q2 : base;
    lim = s2 ? n2 + GR * q2 : lim;
    base = s3 ? b3 - GR * q3 : base;
    lim = s3 ? n3 + GR * q3 : lim;
    const bool ok = lane < e_np;
    e_ra = ok ? base + GR * lane : b0;  // lanes past the quad's groups keep a valid row
    if (D3 == 8) {
      const bool has1 = ok && 2 * lane + 1 < lim;
      e_ia = uniq_i3[e_ra];
      e_ib = uniq_i3[has1 ? e_ra + 1 : e_ra];
      e_jh = (j << 16) | (has1 ? 1 << 18 : 0);
    } else {
      const int left = lim - GR * lane;
      const int cnt = ok ? (left < GR ? left : GR) : 1;
      // the quad's row list: slice j's rows at positions p_j .. p_j + n_j - 1
      const int p1 = n0, p2 = p1 + n1, p3 = p2 + n2, ptot = p3 + n3;
      auto list_row = [&](int x) {  // row at position x (x < ptot), else a valid row
        const bool t1 = x >= p1, t2 = x >= p2, t3 = x >= p3;
        int r = b0 + x;
        r = t1 ? b1 + x - p1 : r;
        r = t2 ? b2 + x - p2 : r;
        r = t3 ? b3 + x - p3 : r;
        return x < ptot ? r : b0;
      };
      e_i3lo = uniq_i3[list_row(lane)];
      e_i3hi = uniq_i3[list_row(lane + 64)];
      int pj = 0, qj = 0;
      pj = s1 ? p1 : pj;
      qj = s1 ? q1 : qj;
      pj = s2 ? p2 : pj;
      qj = s2 ? q2 : qj;
      pj = s3 ? p3 : pj;
      qj = s3 ? q3 : qj;
      e_ia = ok ? pj + GR * (lane - qj) : 0;
      e_ib = 0;
      e_jh = (j << 16) | ((cnt - 1) << 19);
    }
  };
  auto pair_load = [&](BwPair& X, int P) {
    const int ra = __builtin_amdgcn_readlane(d_ra, P), pk = __builtin_amdgcn_readlane(d_pk, P);
    X.j = (pk >> 16) & 3;
    if (D3 == 8) {
      const int i3a = pk & 255, i3b = (pk >> 8) & 255;
      const bool has1 = (pk >> 18) & 1;
      // rows ra and ra + 1 through one descriptor that ends after the rows that exist
      const buf_t eb = make_buf(dE + (size_t)(uint32_t)ra * 128, has1 ? 1024u : 512u);
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) X.eb[s4] = buf_f32(eb, vo_eb, 128u * s4);
      X.e4 = buf_f32x4(eb, vo_e4);
      X.d4 = buf_f32x4(g3buf, vo_d4 + (uint32_t)(prow ? i3b : i3a) * 1024u);
      const int i3z = i3a > 0 ? i3a - 1 : (s.n3 > 1 ? 1 : 0);
      X.i3m = rowsel ? (has1 ? i3b : i3z) : i3a;
    } else {
      const int x0 = pk & 255, cnt = ((pk >> 19) & 7) + 1;
      // the group's rows through one descriptor that ends after its last real row
      const buf_t eb = make_buf(dE + (size_t)(uint32_t)ra * DW, (uint32_t)cnt * (4u * DW));
      const float4 v = buf_f32x4(eb, vo_eb);
      X.eb[0] = v.x;
      X.eb[1] = v.y;
      X.eb[2] = v.z;
      X.eb[3] = v.w;
      const float2 e0 = buf_f32x2(eb, vo_e4), e1 = buf_f32x2(eb, vo_e4 + 4u * DW);
      X.e4 = make_float4(e0.x, e0.y, e1.x, e1.y);
      // i3 of group row k (rows past the last real one repeat it), from the lane of the
      // row list that holds it (a cross-lane read: every call runs on all lanes)
      auto i3_at = [&](int k) {
        const int x = x0 + (k < cnt ? k : cnt - 1);
        const int lo = __builtin_amdgcn_ds_bpermute(4 * x, d_i3lo), hi = __builtin_amdgcn_ds_bpermute(4 * x, d_i3hi);
        return x < 64 ? lo : hi;
      };
      const int r0 = i3_at(2 * l4), r1 = i3_at(2 * l4 + 1);
      const float2 g0 = buf_f32x2(g3buf, vo_d4 + (uint32_t)r0 * (128u * D3));
      const float2 g1 = buf_f32x2(g3buf, vo_d4 + (uint32_t)r1 * (128u * D3));
      X.d4 = make_float4(g0.x, g0.y, g1.x, g1.y);
      // read on every lane, outside the select: a lane whose own row is missing can
      // still hold a list entry that another lane's row needs
      const int ia = i3_at(asel);
      X.i3m = asel < cnt ? ia : s.n3 + asel;
    }
  };

  int f = 0, ns = 0, run = -1;
  // claim a chunk; load its slice descriptors and the i3 words of its first quad
  // static modes: this wave's fixed share of the owner's chunks, in order
  const int owid = (blockIdx.x / nq) * BW_WAVES + wave, onw = (gridDim.x / nq) * BW_WAVES;
  int st_next = share_lo(nch, onw, owid);
  const int st_hi = share_lo(nch, onw, owid + 1);
  auto next_chunk = [&]() {
    const int cc = sched_static(s.sched) ? (st_next < st_hi ? st_next++ : -1) : claim_queues(qctr, nch, 1, 0, &cursor);
    if (cc >= 0) {
      const int4 ch = chunks[c_lo + cc];
      f = __builtin_amdgcn_readfirstlane(ch.x);
      ns = __builtin_amdgcn_readfirstlane(ch.y);
      run = __builtin_amdgcn_readfirstlane(ch.z);
      const int sl = f + (lane < ns ? lane : 0);
      const int4 sd = slices[sl];
      c_rb = sd.y;
      c_nr = lane < ns ? sd.z - sd.y : 0;
      c_i1 = slice_i1[sl];
      build_desc(0);
    }
    qd = 0;
    return cc;
  };
  // The LDS accumulate of the last row pair: its two swaps (expected words pa_e,
  // returned old words pa_o, added values pa_v).  A swap took place when the old
  // word equals the expected one; otherwise it is retried from the returned word.
  // Checking at the next pair lets the round trip overlap that pair's products,
  // and a retry before the next pair's swaps keeps every add.
  uint64_t* pa_u = reinterpret_cast<uint64_t*>(g3acc);
  uint64_t pa_e0 = 0, pa_e1 = 0, pa_o0 = 0, pa_o1 = 0;
  f32x4 pa_v = {0.f, 0.f, 0.f, 0.f};
  auto acc_finish = [&]() {
    bool d0 = pa_o0 == pa_e0, d1 = pa_o1 == pa_e1;
    while (!(d0 && d1)) {
      if (!d0) {
        pa_e0 = pa_o0;
        pa_o0 = lds_cas_old(pa_u, pa_e0, add2(pa_e0, pa_v[0], pa_v[1]));
        d0 = pa_o0 == pa_e0;
      }
      if (!d1) {
        pa_e1 = pa_o1;
        pa_o1 = lds_cas_old(pa_u + 1, pa_e1, add2(pa_e1, pa_v[2], pa_v[3]));
        d1 = pa_o1 == pa_e1;
      }
    }
  };
  // The next quad's operands are loaded before the current quad's dA product, so
  // that product and its stores cover their latency: its row-pair descriptors,
  // its stage-1 A operand and its first two row pairs.  At a chunk end the next
  // chunk is claimed first.  In a quad of fewer than four slices the missing
  // slices' A rows repeat a loaded slice: a product's output row depends on its own
  // operand row only, and the stack rows of missing slices are neither read by the
  // row pairs nor summed into dB nor stored as dA, so they need no clearing.
  float Aop[8];
  float ATq[8];  // dB A operands A_j^T of the quad's four slices, (j, half) -> 2 j + half
  BwPair XA, XB, XC;
  auto prefetch_quad = [&]() {
    d_ra = e_ra;
    d_pk = e_ia | (e_ib << 8) | e_jh;
    d_i3lo = e_i3lo;
    d_i3hi = e_i3hi;
    np = e_np;
    if (qd + 4 < ns) build_desc(qd + 4);  // the quad after it, one quad ahead
    const int nq4 = ns - qd < 4 ? ns - qd : 4;
    const int aj = l15 >> 2;
    const int i1a = __builtin_amdgcn_readlane(c_i1, qd), i1b = __builtin_amdgcn_readlane(c_i1, qd + 1);
    const int i1c = __builtin_amdgcn_readlane(c_i1, qd + 2), i1d = __builtin_amdgcn_readlane(c_i1, qd + 3);
    const float* Ag = G1t + (uint32_t)sel4(aj < nq4 ? aj : 0, i1a, i1b, i1c, i1d) * 128u +
                      (uint32_t)((lane & 3) * 32 + l4);
#pragma unroll
    for (int s4 = 0; s4 < 8; ++s4) Aop[s4] = Ag[4 * s4];
    // loaded with Aop, ahead of every row-pair load of the quad: vector memory
    // counts complete in issue order, so a wait for an operand loaded later (at a
    // slice switch) would also wait for the row pairs prefetched before it
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float* Aj = G1t + (uint32_t)__builtin_amdgcn_readlane(c_i1, qd + j) * 128u + (uint32_t)(l4 * 32 + l15);
      ATq[2 * j] = Aj[0];
      ATq[2 * j + 1] = Aj[16];
    }
    pair_load(XA, 0);
    pair_load(XB, np > 1 ? 1 : 0);
  };
  int c = next_chunk();
  if (c >= 0) prefetch_quad();
  while (c >= 0) {
    if (run != cur_run) {
      const float* Bg = G2 + (uint32_t)run * 4096u + 16 * h;
#pragma unroll
      for (int s4 = 0; s4 < 8; ++s4)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) Bop[4 * s4 + nt] = Bg[((4 * s4 + l4) * 4 + nt) * 32 + l15];
#pragma unroll
      for (int nt2 = 0; nt2 < 2; ++nt2)
#pragma unroll
        for (int q = 0; q < 4; ++q) {  // B_h[a][j2 = l4][b' = 4 q .. 4 q + 3]: 16 contiguous bytes
          const float4 v = *(const float4*)(Bg + ((16 * nt2 + l15) * 4 + l4) * 32 + 4 * q);
          BTop[16 * nt2 + 4 * q + 0] = v.x;
          BTop[16 * nt2 + 4 * q + 1] = v.y;
          BTop[16 * nt2 + 4 * q + 2] = v.z;
          BTop[16 * nt2 + 4 * q + 3] = v.w;
        }
      cur_run = run;
    }
    const int nqs = ns - qd < 4 ? ns - qd : 4;
    const int sb = f + qd;
    // stage 1: Cstack_h (16 x 64) = Astack (16 x 32) . B_h (32 x 64),
    // Astack[(slice aj, j1 = lane & 3)][a = 4 s + l4] (rows of missing slices unused)
    {
      f32x4 Cs[4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) Cs[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s4 = 0; s4 < 8; ++s4) {
        const float a = Aop[s4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) Cs[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Bop[4 * s4 + nt], Cs[nt], 0, 0, 0);
      }
      // lane holds C_h[slice l4][j1 r][j2 nt][b' l15]: row 4 l4 + r, column 16 nt + l15
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) scr_c[SCR_PITCH * r + 16 * nt] = Cs[nt][r];
      wave_lds_sync();
    }
    // per slice: dD A operand C_h^T[b' = l15][(j1 j2) = 4 s + l4] (d3 = 8) or
    // C_h^T[b' = l15][(j1 j2) = 4 l4 + s] (d3 = 2)
    float CT[4];
    auto slice_begin = [&](int j) {
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) {
        if (D3 == 8)
          CT[s4] = scr[4 * SCR_PITCH * j + SCR_PITCH * s4 + lane];  // row 4 j + s4
        else
          CT[s4] = scr[4 * SCR_PITCH * j + SCR_PITCH * l4 + 16 * s4 + l15];  // row 4 j + l4
      }
    };
    slice_begin(0);
    f32x4 dC = {0.f, 0.f, 0.f, 0.f};
    auto pair_compute = [&](const BwPair& X) {
      // this lane's accumulator words, read before the products so the read's
      // latency overlaps them
      float* ap = g3acc + (uint32_t)X.i3m * APITCH + o_g3;
      const ulonglong2 w = *reinterpret_cast<const ulonglong2*>(ap);
      float ebk[4];
      if (D3 == 8) {
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) ebk[s4] = X.eb[s4];
      } else {
        // dE[row][(4 l4 + s) * 2 + j3]: the even lane holds s = 0, 1 of both j3, the odd
        // lane s = 2, 3; each keeps its own j3 and takes the rest from its neighbour.
        // The swaps run on every lane before the selects: inside a conditional they
        // would run under a partial lane mask, where a neighbour's value is not read
        const float w0 = swap_neighbour(X.eb[0]), w1 = swap_neighbour(X.eb[1]);
        const float w2 = swap_neighbour(X.eb[2]), w3 = swap_neighbour(X.eb[3]);
        ebk[0] = odd_lane ? w1 : X.eb[0];
        ebk[1] = odd_lane ? w3 : X.eb[2];
        ebk[2] = odd_lane ? X.eb[1] : w0;
        ebk[3] = odd_lane ? X.eb[3] : w2;
      }
      f32x4 dd = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) dd = __builtin_amdgcn_mfma_f32_16x16x4f32(CT[s4], ebk[s4], dd, 0, 0, 0);
      dC = __builtin_amdgcn_mfma_f32_16x16x4f32(X.e4.x, X.d4.x, dC, 0, 0, 0);
      dC = __builtin_amdgcn_mfma_f32_16x16x4f32(X.e4.y, X.d4.y, dC, 0, 0, 0);
      dC = __builtin_amdgcn_mfma_f32_16x16x4f32(X.e4.z, X.d4.z, dC, 0, 0, 0);
      dC = __builtin_amdgcn_mfma_f32_16x16x4f32(X.e4.w, X.d4.w, dC, 0, 0, 0);
      // dd: lane holds dD_h[b' = 4 l4 + r][group row l15 / d3][j3 = l15 % d3]
      // every lane swaps (the zero row's column adds exact zeros), so the add is
      // straight-line code and the read stays ahead of the products; the previous
      // pair's swaps are checked first, this pair's at the next pair
      acc_finish();
      pa_u = reinterpret_cast<uint64_t*>(ap);
      pa_e0 = w.x;
      pa_e1 = w.y;
      pa_v = dd;
      pa_o0 = lds_cas_old(pa_u, w.x, add2(w.x, dd[0], dd[1]));
      pa_o1 = lds_cas_old(pa_u + 1, w.y, add2(w.y, dd[2], dd[3]));
    };
    // slice j done: dC_h to rows 4 j .. 4 j + 3 of the stack, for the quad's dB and dA
    auto slice_end = [&](int j) {
      wave_lds_sync();
#pragma unroll
      for (int r = 0; r < 4; ++r) scr_d[4 * SCR_PITCH * j + 16 * r] = dC[r];  // row 4 j + l4, column 16 r + l15
      dC = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    // row pairs of the quad in order, three per iteration over three operand
    // sets: the operands of the next two pairs are always in flight while one is
    // computed (indices clamped, so every load is unconditional and in bounds)
    int cj = 0;
    auto step = [&](const BwPair& X) {
      if (X.j != cj) {
        slice_end(cj);
        slice_begin(X.j);
        cj = X.j;
      }
      pair_compute(X);
    };
    for (int P = 0; P < np; P += 3) {
      pair_load(XC, P + 2 < np ? P + 2 : np - 1);
      step(XA);
      pair_load(XA, P + 3 < np ? P + 3 : np - 1);
      if (P + 1 < np) step(XB);
      pair_load(XB, P + 4 < np ? P + 4 : np - 1);
      if (P + 2 < np) step(XC);
    }
    slice_end(cj);
    wave_lds_sync();
    // dB_h += A_j^T . dC_j (M = a, N = (j2, b'), K = j1) for the quad's slices, before
    // the next quad's operands replace ATq; each lane's B operand dC_j[j1 = l4][16 nt + l15]
    // is what it wrote to the stack itself
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j < nqs) {
        float dcj[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) dcj[nt] = scr_d[4 * SCR_PITCH * j + 16 * nt];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          dB[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(ATq[2 * j], dcj[nt], dB[nt], 0, 0, 0);
          dB[4 + nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(ATq[2 * j + 1], dcj[nt], dB[4 + nt], 0, 0, 0);
        }
      }
    }
    // the next quad: the rest of this chunk, or the first quad of the next chunk
    const int c_done = c;
    const bool chunk_end = qd + 4 >= ns;
    if (chunk_end)
      c = next_chunk();
    else
      qd += 4;
    // one call site, so the loads land in the registers the next quad reads (two
    // inlined copies would need register copies, and so waits, where they merge)
    if (c >= 0) prefetch_quad();
    // dA_h (16 x 32) = dCstack_h (16 x 64) . B_h^T (64 x 32), the contraction over
    // (j2, b') taken as (j2 = l4, b' = s) in step s, so that each lane reads 16
    // contiguous floats of its stack row l15
    {
      f32x4 dA0 = {0.f, 0.f, 0.f, 0.f}, dA1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(scr_a + 4 * q);
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const float av = v[c4];
          dA0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av, BTop[4 * q + c4], dA0, 0, 0, 0);
          dA1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av, BTop[16 + 4 * q + c4], dA1, 0, 0, 0);
        }
      }
      // lane holds dA_h[slice l4][j1 r][a = 16 nt2 + l15]; the partial is read once, by the
      // dG1 sum: stored non-temporally
      if (l4 < nqs) {
        float* dst = dApart + ((size_t)h * nsl_cap + (sb + l4)) * 128 + l15;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          __builtin_nontemporal_store(dA0[r], dst + r * 32);
          __builtin_nontemporal_store(dA1[r], dst + r * 32 + 16);
        }
      }
    }
    wave_lds_sync();
    if (chunk_end) {
      // dB_h partial of the finished chunk, lane holds dB_h[a = 16 mt + 4 l4 + r][(j2 = nt, b' = l15)];
      // read once, by the dG2 sum: stored non-temporally
      float* dst = dBpart + ((size_t)h * nch_cap + (c_lo + c_done)) * 2048;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            __builtin_nontemporal_store(dB[4 * mt + nt][r], dst + (16 * mt + 4 * l4 + r) * 64 + 16 * nt + l15);
#pragma unroll
      for (int k = 0; k < 8; ++k) dB[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
  acc_finish();
  __syncthreads();
  float* gdst = g3part + (size_t)blockIdx.x * acc_n;  // the table's rows only
  for (int i = threadIdx.x; i < acc_n; i += blockDim.x) gdst[i] = g3acc[(i / AROW) * APITCH + i % AROW];
}

// Each reduction writes its sum into `out` (the gradient), or with lr given,
// subtracts lr times the sum from `out` (the core itself: the update of the fused
// backward-and-SGD call).  Every element of its core is visited exactly once.
__device__ __forceinline__ void put_grad(float* out, int64_t i, float acc, float lr, bool update) {
  out[i] = update ? out[i] - lr * acc : acc;
}

// dG1[t][i1] = sum over i2 of the dA halves of the slices of prefix (i1, i2).
// The block lists the slices of (t, i1) in i2 order (512 prefixes per round,
// the list G1_LIST entries at a time), and its eight waves take list entries
// g, g + 8, ... (two columns per lane, eight 8-byte loads in flight); the wave
// sums are combined in a fixed order.
constexpr int G1_LIST = 4096;

constexpr int RED_THREADS = 512;

__device__ __forceinline__ void reduce_g1(int ti1, ShapeArgs s, const uint32_t* __restrict__ dense_cnt,
                                          const uint32_t* __restrict__ dense_base,
                                          const float* __restrict__ dApart, int nsl_cap, float* __restrict__ dG1,
                                          float lr, bool update) {
  __shared__ int list[G1_LIST];
  __shared__ uint32_t wsum[8];
  __shared__ float2 red[8][64];
  // ti1 = t * n1 + i1
  const int t = ti1 / s.n1, i1 = ti1 % s.n1;
  const int g = threadIdx.x >> 6, e = threadIdx.x & 63;  // eight waves, two columns per lane
  const float2* P0 = reinterpret_cast<const float2*>(dApart) + e;
  const float2* P1 = reinterpret_cast<const float2*>(dApart + (size_t)nsl_cap * 128) + e;
  float2 a[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) a[k] = make_float2(0.f, 0.f);
  auto add = [](float2& x, const float2 y) {
    x.x += y.x;
    x.y += y.y;
  };
  for (int i2b = 0; i2b < s.n2; i2b += 512) {
    const int i2 = i2b + (int)threadIdx.x;
    uint32_t cnt = 0, base = 0;
    if (i2 < s.n2) {
      const int64_t slot = ((int64_t)t * s.n2 + i2) * s.n1 + i1;
      cnt = dense_cnt[slot];
      base = dense_base[slot];
    }
    uint32_t total;
    const uint32_t pos = block_excl_scan<uint32_t, 512>(cnt, wsum, &total);
    // the round's slice list, G1_LIST entries at a time; wave g takes entries g, g + 8, ...
    for (uint32_t w0 = 0; w0 < total; w0 += G1_LIST) {
      const uint32_t k0 = w0 > pos ? w0 - pos : 0u, k1e = w0 + G1_LIST - pos;
      const uint32_t k1 = pos >= w0 + G1_LIST ? 0u : (cnt < k1e ? cnt : k1e);
      for (uint32_t k = k0; k < k1; ++k) list[pos + k - w0] = (int)(base + k);
      __syncthreads();
      const int wn = (int)(total - w0 < (uint32_t)G1_LIST ? total - w0 : (uint32_t)G1_LIST);
      int j = g;
      for (; j + 56 < wn; j += 64) {  // sixteen loads in flight; the same accumulators in the same order
        float2 v[16];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const size_t l = (size_t)list[j + 8 * q] * 64;
          v[2 * q] = ntl2(P0 + l);
          v[2 * q + 1] = ntl2(P1 + l);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          add(a[2 * (q & 3)], v[2 * q]);
          add(a[2 * (q & 3) + 1], v[2 * q + 1]);
        }
      }
      for (; j + 24 < wn; j += 32) {
        const size_t l0 = (size_t)list[j] * 64, l1 = (size_t)list[j + 8] * 64;
        const size_t l2 = (size_t)list[j + 16] * 64, l3 = (size_t)list[j + 24] * 64;
        add(a[0], ntl2(P0 + l0));
        add(a[1], ntl2(P1 + l0));
        add(a[2], ntl2(P0 + l1));
        add(a[3], ntl2(P1 + l1));
        add(a[4], ntl2(P0 + l2));
        add(a[5], ntl2(P1 + l2));
        add(a[6], ntl2(P0 + l3));
        add(a[7], ntl2(P1 + l3));
      }
      for (; j < wn; j += 8) {
        const size_t l0 = (size_t)list[j] * 64;
        add(a[0], ntl2(P0 + l0));
        add(a[1], ntl2(P1 + l0));
      }
      __syncthreads();
    }
  }
  float2 r;
  r.x = ((a[0].x + a[1].x) + (a[2].x + a[3].x)) + ((a[4].x + a[5].x) + (a[6].x + a[7].x));
  r.y = ((a[0].y + a[1].y) + (a[2].y + a[3].y)) + ((a[4].y + a[5].y) + (a[6].y + a[7].y));
  red[g][e] = r;
  __syncthreads();
  if (g == 0) {
    float2 v = red[0][e];
#pragma unroll
    for (int k = 1; k < 8; ++k) add(v, red[k][e]);
    put_grad(dG1, (int64_t)ti1 * 128 + 2 * e, v.x, lr, update);
    put_grad(dG1, (int64_t)ti1 * 128 + 2 * e + 1, v.y, lr, update);
  }
}

// dG2[t][i2][a][j2][16 h + b'] = sum of the chunk partials of run (t, i2), half h
// (rh = 2 run + h)
__device__ __forceinline__ void reduce_g2(int rh, const uint32_t* __restrict__ run_base,
                                          const float* __restrict__ dBpart, int nch_cap, float* __restrict__ dG2,
                                          float lr, bool update) {
  const int run = rh >> 1, h = rh & 1;
  const int c0 = (int)run_base[run], c1 = (int)run_base[run + 1];
  // thread k owns elements k + 512 m (m < 4); four chunks' loads are in flight
  // together and added in chunk order
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  const float* src = dBpart + ((size_t)h * nch_cap + c0) * 2048 + threadIdx.x;
  int c = c0;
  for (; c + 4 <= c1; c += 4, src += 4 * 2048) {
    float v[4][4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int m = 0; m < 4; ++m) v[k][m] = ntl(src + k * 2048 + RED_THREADS * m);
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int m = 0; m < 4; ++m) acc[m] += v[k][m];
  }
  for (; c < c1; ++c, src += 2048) {
#pragma unroll
    for (int m = 0; m < 4; ++m) acc[m] += ntl(src + RED_THREADS * m);
  }
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int e = (int)threadIdx.x + RED_THREADS * m;
    const int a = e >> 6, j2 = (e >> 4) & 3, bp = e & 15;
    put_grad(dG2, (int64_t)run * 4096 + (a * 4 + j2) * 32 + 16 * h + bp, acc[m], lr, update);
  }
}

// dG3[t][i3][16 h + b'][j3] = sum over the workgroups that owned (t, h); block xb of
// owner q covers accumulator elements [512 xb, 512 xb + 512)
template <int D3>
__device__ __forceinline__ void reduce_g3(int q, int xb, ShapeArgs s, const float* __restrict__ g3part, int nwg,
                                          float* __restrict__ dG3, float lr, bool update) {
  const int nq = 2 * s.T;
  const int t = q % s.T, h = q / s.T;
  const int acc_n = s.n3 * 16 * D3;
  const int e = xb * RED_THREADS + threadIdx.x;
  if (e >= acc_n) return;
  // four independent sums, so that four loads are in flight
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  int w = q;
  for (; w + 3 * nq < nwg; w += 4 * nq) {
    a0 += ntl(g3part + (int64_t)w * acc_n + e);
    a1 += ntl(g3part + (int64_t)(w + nq) * acc_n + e);
    a2 += ntl(g3part + (int64_t)(w + 2 * nq) * acc_n + e);
    a3 += ntl(g3part + (int64_t)(w + 3 * nq) * acc_n + e);
  }
  for (; w < nwg; w += nq) a0 += ntl(g3part + (int64_t)w * acc_n + e);
  const float acc = (a0 + a1) + (a2 + a3);
  const int i3 = e / (16 * D3), j3 = (e >> 4) % D3, bp = g3_unslot(j3, e & 15);
  put_grad(dG3, (((int64_t)t * s.n3 + i3) * 32 + 16 * h + bp) * D3 + j3, acc, lr, update);
}

// The three reductions in one launch, so they overlap: the first blocks reduce dG3
// (few blocks, each a chain of one load per owner workgroup), the next T n1 dG1,
// the rest (2 T n2) dG2.
template <int D3>
__global__ void __launch_bounds__(RED_THREADS) k_reduce_grads(ShapeArgs s, const uint32_t* __restrict__ dense_cnt,
                                                              const uint32_t* __restrict__ dense_base,
                                                              const float* __restrict__ dApart, int nsl_cap,
                                                              const uint32_t* __restrict__ run_base,
                                                              const float* __restrict__ dBpart, int nch_cap,
                                                              const float* __restrict__ g3part, int nwg,
                                                              float* __restrict__ dG1, float* __restrict__ dG2,
                                                              float* __restrict__ dG3, float lr, bool update) {
  const int b = blockIdx.x;
  const int per_q = (s.n3 * 16 * D3 + RED_THREADS - 1) / RED_THREADS;
  const int n3b = 2 * s.T * per_q, n1b = s.T * s.n1;
  if (b < n3b) {
    reduce_g3<D3>(b / per_q, b % per_q, s, g3part, nwg, dG3, lr, update);
  } else if (b < n3b + n1b) {
    reduce_g1(b - n3b, s, dense_cnt, dense_base, dApart, nsl_cap, dG1, lr, update);
  } else {
    reduce_g2(b - n3b - n1b, run_base, dBpart, nch_cap, dG2, lr, update);
  }
}

bool bwd_r32_supported(const Shape& s, int64_t max_indices) {
  // d = (4, 4, 8) or (4, 4, 2); 32-bit float offsets into dE (rows x at most 128), G1 (slices of 128),
  // G2 (slices of 4,096) and G3 (slices of at most 256) must fit
  // LDS: the n3 x 128 accumulator plus 8 x 16 x SCR_PITCH scratch floats fit 160 KB for n3 <= 252
  // (d3 = 8); i3 travels in 8 bits (d3 = 8) and the row list of d3 = 2 keeps the same bound
  return s.d1 == 4 && s.d2 == 4 && (s.d3 == 8 || s.d3 == 2) && s.R == 32 && s.n3 <= 252 && s.T <= 64 &&
         max_indices * 128 < (int64_t(1) << 31) && (int64_t)s.T * s.n3 * 256 < (int64_t(1) << 31) &&
         (int64_t)s.T * s.n1 * 128 < (int64_t(1) << 31) && (int64_t)s.T * s.n2 * 4096 < (int64_t(1) << 31);
}

// With update set, dG1..dG3 are the cores themselves and receive G -= lr * dG.
hipError_t launch_bwd_r32(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                          float* dG1, float* dG2, float* dG3, float lr, bool update, const Prof& prof,
                          hipStream_t st) {
  const int nq = 2 * s.T;
  const int cap = persistent_grid() < MAX_BWD_WG ? persistent_grid() : MAX_BWD_WG;
  int per_q = cap / nq;
  if (per_q < 1) per_q = 1;
  const int grid = nq * per_q;
  if (grid > MAX_BWD_WG || nq * SCHED_STRIDE > C_TOTAL - C_BWD_CTR) return hipErrorInvalidValue;
  hipError_t e = fill_u32(reinterpret_cast<uint32_t*>(w.ctr + C_BWD_CTR), nq * SCHED_STRIDE, 0u, st);
  if (e != hipSuccess) return e;
  const bool d8 = s.d3 == 8;
  const size_t lds = sizeof(float) * (d8 ? (size_t)s.n3 * 128 : (size_t)(s.n3 + 8) * 36) + sizeof(float) * BW_WAVES * BW_SCR;
  const void* kfn = d8 ? (const void*)k_bwd_r32<8> : (const void*)k_bwd_r32<2>;
  e = hipFuncSetAttribute(kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  prof_begin(prof, K_BWD_FUSED, st);
  hipLaunchKernelGGL(d8 ? k_bwd_r32<8> : k_bwd_r32<2>, dim3(grid), dim3(64 * BW_WAVES), lds, st, shape_args(s), G1, G2, G3,
                     (const float*)w.E, (const int4*)w.slices, (const int32_t*)w.slice_i1, (const int4*)w.chunks,
                     (const uint32_t*)w.run_nch, (const int32_t*)w.uniq_i3, w.ctr, w.dApart, w.dBpart, w.g3part,
                     (int)w.nsl_max, (int)w.nch_max);
  prof_end(prof, K_BWD_FUSED, st);
  const int red_blocks = s.T * s.n1 + 2 * s.T * s.n2 + nq * ((s.n3 * 16 * s.d3 + RED_THREADS - 1) / RED_THREADS);
  hipLaunchKernelGGL(d8 ? k_reduce_grads<8> : k_reduce_grads<2>, dim3(red_blocks), dim3(RED_THREADS), 0, st, shape_args(s),
                     (const uint32_t*)w.dense_cnt, (const uint32_t*)w.dense_base, (const float*)w.dApart,
                     (int)w.nsl_max, (const uint32_t*)w.run_nch, (const float*)w.dBpart, (int)w.nch_max,
                     (const float*)w.g3part, grid, dG1, dG2, dG3, lr, update);
  return hipGetLastError();
}

}  // namespace ttemb
