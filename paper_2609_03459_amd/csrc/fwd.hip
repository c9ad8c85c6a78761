// Forward pass of the TT-embedding gather (FlowTT Section 3.2, Fig. 3).
//   fused kernel : per work slice (rows of one prefix group), C = A.B is built
//                  once in LDS and reused for every row: E_u = C.D_u
//   pooling      : V[bag] = sum of E over the bag's occurrences, in order
// Slices come in (table, i2, i1) order so consecutive groups share G2[i2].
#include "common.h"

namespace ttemb {

ShapeArgs shape_args(const Shape& s) {
  ShapeArgs a;
  a.T = s.T;
  a.n1 = s.n1;
  a.n2 = s.n2;
  a.n3 = s.n3;
  a.d1 = s.d1;
  a.d2 = s.d2;
  a.d3 = s.d3;
  a.R = s.R;
  a.D = s.D;
  a.n12 = s.n12;
  a.Npad = s.Npad;
  a.sched = s.sched;
  return a;
}

constexpr int FWD_LDS_FLOATS = 40448;    // dynamic LDS budget (158 KB of the 160 KB)
constexpr int FWD_CHUNK = 8;             // slices per claim

// sum over k < n of x[k * xs] * y[k * ys], four independent partial sums
__device__ __forceinline__ float fdot_strided(const float* x, int xs, const float* y, int ys, int n) {
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

// Generic fused forward for any shape within the library limits (plain VALU).  A
// block claims FWD_CHUNK consecutive slices; B = G2[t][i2] of their (t, i2) run is
// staged in LDS (rows padded by one float) when it fits, again whenever the run
// changes; per slice A is staged, C = A.B is built once per prefix group and
// E = C.D per row.
// FWD_THREADS = 1024 (sixteen waves: latency hiding at one block per CU) for large
// products, 256 for small ones (where a block's barriers dominate)
template <int FWD_THREADS>
__global__ void __launch_bounds__(FWD_THREADS) k_fwd_generic(ShapeArgs s, const float* __restrict__ G1,
                                                             const float* __restrict__ G2,
                                                             const float* __restrict__ G3,
                                                             const int4* __restrict__ slices,
                                                             const int4* __restrict__ chunks,
                                                             const uint32_t* __restrict__ run_base,
                                                             const int32_t* __restrict__ uniq_i3,
                                                             int32_t* __restrict__ ctr, float* __restrict__ E,
                                                             float* __restrict__ ckpt, int32_t* __restrict__ ckpt_tag,
                                                             int stage_b) {
  extern __shared__ float lds[];
  const int d2R = s.d2 * s.R;
  const int nC = s.d1 * d2R;
  const int nB = s.R * d2R;
  const int bp = stage_b ? d2R + 1 : d2R;
  float* C = lds;            // nC = d1 * d2 * R
  float* As = C + nC;        // d1 * R
  float* Bs = As + s.d1 * s.R;  // R * (d2R + 1) when stage_b
  __shared__ int s_chunk, s_flag;
  const int nsl = ctr[C_NSLICES];
  // work units: FWD_CHUNK consecutive slices, or with SCHED_GROUP the chunk list's whole groups
  const bool by_group = s.sched == SCHED_GROUP;
  const int nchunks = by_group ? (int)run_base[s.T * s.n2] : (nsl + FWD_CHUNK - 1) / FWD_CHUNK;
  int victim = 0;
  int next = share_lo(nchunks, (int)gridDim.x, (int)blockIdx.x);
  int cur_pg = -1, cur_run = -1;
  const float* Bm = G2;
  while (true) {
    const int c = claim_block_sched(s.sched, ctr + C_FWD_CTR, nchunks, blockIdx.x % SCHED_NQ, &victim, &s_chunk,
                                    &next);
    if (c < 0) break;
    int s0, s1;
    if (by_group) {
      const int4 ch = chunks[c];
      s0 = ch.x;
      s1 = ch.x + ch.y;
    } else {
      s0 = c * FWD_CHUNK;
      s1 = s0 + FWD_CHUNK < nsl ? s0 + FWD_CHUNK : nsl;
    }
    for (int si = s0; si < s1; ++si) {
      const int4 sl = slices[si];
      const int p = sl.x, rb = sl.y, re = sl.z;
      const uint32_t key = (uint32_t)sl.w;
      const int t = (int)(key / (uint32_t)s.n12), q = (int)(key % (uint32_t)s.n12);
      const int i1 = q / s.n2, run = t * s.n2 + q % s.n2;
      if (p != cur_pg) {
        // intermediate C = A.B, kept in LDS while rows of this group follow; with
        // the checkpoint, reloaded if another block published it, and published if
        // the group goes on past this claim (where a stealing block may meet it)
        __syncthreads();  // the previous slice's rows are done with C
        const bool ck = s.sched == SCHED_STEAL_CKPT;
        if (!(ck && ckpt_load(ckpt, ckpt_tag, p, C, nC, &s_flag))) {
          const float* Bg = G2 + (int64_t)run * nB;
          if (run != cur_run) {
            if (stage_b)
              for (int o = threadIdx.x; o < nB; o += FWD_THREADS) {
                const int a = o / d2R, cc = o - a * d2R;
                Bs[a * bp + cc] = Bg[o];
              }
            Bm = stage_b ? Bs : Bg;
            cur_run = run;
          }
          const float* Ag = G1 + ((int64_t)(t * s.n1 + i1) * s.d1) * s.R;
          for (int o = threadIdx.x; o < s.d1 * s.R; o += FWD_THREADS) As[o] = Ag[o];
          __syncthreads();
          for (int o = threadIdx.x; o < nC; o += FWD_THREADS) {
            const int j1 = o / d2R, cc = o - j1 * d2R;
            C[o] = fdot_strided(As + j1 * s.R, 1, Bm + cc, bp, s.R);
          }
          if (ck && s1 < nsl && slices[s1].x == p) {  // the group goes on past this claim
            __syncthreads();
            ckpt_store(ckpt, ckpt_tag, p, C, nC, &s_flag);
          }
        }
        __syncthreads();
        cur_pg = p;
      }
      // embedding rows E_u = C . D_u, C viewed as (d1 d2) x R
      const int total = (re - rb) * s.D;
      for (int o = threadIdx.x; o < total; o += FWD_THREADS) {
        const int r = o / s.D, j = o - r * s.D;
        const int u = rb + r;
        const int i3 = uniq_i3[u];
        const int jr = j / s.d3, j3 = j - jr * s.d3;
        const float* Dm = G3 + (int64_t)(t * s.n3 + i3) * s.R * s.d3 + j3;
        E[(int64_t)u * s.D + j] = fdot_strided(C + jr * s.R, 1, Dm, s.d3, s.R);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// MFMA forward for d = (4, 4, 8), R = 32 (D = 128).  Persistent waves claim
// chunks (up to 32 slices of one (t, i2) run, so B = G2[t][i2] stays in VGPRs)
// and work through them four slices ("a quad") at a time:
//   * stage 1: Cstack (16 x 128) = Astack (16 x 32) . B (32 x 128) with
//     v_mfma_f32_16x16x4f32, rows (slice, j1), columns (j2, b); 64 instructions;
//   * Cstack goes through a per-wave padded LDS tile into the B operand of
//     stage 2, C'^T (b x jj) of one slice;
//   * stage 2 per row pair: E^T (rows x j3, jj) = D^T . C'^T, 8 instructions;
//     each lane ends up with four consecutive floats of one E row (one 16-byte
//     store).
// The next row pair's G3 operands are in flight while a pair is computed.
// ---------------------------------------------------------------------------
constexpr int F32_WAVES = 4;
constexpr int F32_WG_PER_CU = 3;  // three workgroups (12 waves, 111 KB LDS) per CU (four spill at 128 VGPRs)
// Per-wave LDS tile of the C stack: row (slice, j1, j2) holds the 32 b values of one
// (j1, j2), rows F32_ROW floats apart, slices F32_SLICE apart.  The padding puts at
// most two lanes on a bank for the stage-1 writes (the four slices of a write land
// 16 banks apart) and for the stage-2 reads (a lane's row pitch of 36 spreads the
// sixteen rows over distinct bank groups), whether the LDS has 32 or 64 banks, and
// makes every access a per-lane base plus an immediate offset.
constexpr int F32_ROW = 36;
constexpr int F32_SLICE = 16 * F32_ROW + 16;
constexpr int F32_SCR = 4 * F32_SLICE;

// D3 = 8: d = (4, 4, 8), row groups of two rows; D3 = 2: d = (4, 4, 2) (D = 32), row groups
// of eight rows, each lane's stage-2 operand from its own row of the group.
template <int D3>
__global__ void __launch_bounds__(64 * F32_WAVES, F32_WG_PER_CU)
    k_fwd_r32(ShapeArgs s, const float* __restrict__ G1, const float* __restrict__ G2, const float* __restrict__ G3,
              const int4* __restrict__ slices, const int32_t* __restrict__ slice_i1,
              const int4* __restrict__ chunks, const uint32_t* __restrict__ run_base,
              const int32_t* __restrict__ uniq_i3, int32_t* __restrict__ ctr, float* __restrict__ E) {
  __shared__ float scr_all[F32_WAVES * F32_SCR];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float* scr = scr_all + wave * F32_SCR;
  // this lane's stage-1 write base (slice l4, b = l15 (+ 16)) and stage-2 read base
  // (row jj = (j1, j2) = l15, b = 4 s + l4 for D3 = 8, b = 8 l4 + s for D3 = 2)
  float* scr_w = scr + F32_SLICE * (lane >> 4) + (lane & 15);
  const float* scr_r = scr + F32_ROW * (lane & 15) + (D3 == 2 ? 8 : 1) * (lane >> 4);
  constexpr int GR = 16 / D3;              // rows per stage-2 group ("pair" below)
  constexpr int DW = 16 * D3;              // floats per E row
  constexpr uint32_t G3ROW = 128u * D3;    // bytes per G3 row (R d3 floats)
  // E rows of all unique rows beyond the last-level cache: stored non-temporally
  const bool e_nt = (uint64_t)(uint32_t)ctr[C_U] * (4u * DW) > STREAM_BYTES;
  const int nch = (int)run_base[s.T * s.n2];
  const int l15 = lane & 15, l4 = lane >> 4;
  // stage-2 A operand: lane m = l15 = (row asel of the group, j3), K index b = 4 s + l4
  // (D3 = 8) or b = 8 l4 + s (D3 = 2)
  const int asel = l15 / D3;
  const bool odd_lane = (lane & 1) != 0;
  // byte offsets: this lane's stage-2 A words in a G3 row and its E store.  D3 = 8: the
  // word b = l4, j3 = l15 % 8, then 16 D3 bytes per K step.  D3 = 2: the lanes of j3 = 0
  // and 1 of a row share the 64 bytes of b = 8 l4 .. 8 l4 + 7 (both j3), the even lane
  // loading the first 32, the odd lane the second.  Output row 4 l4 + r of the MFMA is
  // group row (4 l4 + r) / D3, so for D3 = 8 four consecutive floats of row l4 / 2, for
  // D3 = 2 two floats of rows 2 l4 and 2 l4 + 1 (the second 128 bytes on)
  const uint32_t vo_d = D3 == 8 ? 4u * (uint32_t)(l4 * D3 + (l15 % D3)) : 4u * (uint32_t)(16 * l4 + 8 * (l15 & 1));
  const uint32_t vo_e = D3 == 8 ? 4u * (uint32_t)((l4 >> 1) * 128 + l15 * 8 + 4 * (l4 & 1))
                                : 4u * (uint32_t)(2 * l4 * DW + l15 * 2);

  int cursor = 0;
  int cur_run = -1;
  float Bop[64];  // B[a = 4 s + l4][16 nt + l15], (s, nt) -> 8 s + nt

  // slice descriptors of the current chunk, lane j holding slice f + j (j < ns;
  // other lanes have no rows): first row, row count, i1
  int c_rb = 0, c_nr = 0, c_i1 = 0;
  int f = 0, ns = 0, run = -1, t = 0, qd = 0;
  int c = -1;
  // static modes: this wave's fixed share of the chunks, in order
  const int wid = blockIdx.x * F32_WAVES + wave, nw = gridDim.x * F32_WAVES;
  int st_next = share_lo(nch, nw, wid);
  const int st_hi = share_lo(nch, nw, wid + 1);
  auto next_chunk = [&]() {
    if (sched_static(s.sched))
      c = st_next < st_hi ? st_next++ : -1;
    else
      c = claim_queues(ctr + C_FWD_CTR, nch, SCHED_NQ, blockIdx.x % SCHED_NQ, &cursor);
    qd = 0;
    if (c >= 0) {
      const int4 ch = chunks[c];
      f = __builtin_amdgcn_readfirstlane(ch.x);
      ns = __builtin_amdgcn_readfirstlane(ch.y);
      run = __builtin_amdgcn_readfirstlane(ch.z);
      t = run / s.n2;
      const int sl = f + (lane < ns ? lane : 0);
      const int4 sd = slices[sl];
      c_rb = sd.y;
      c_nr = lane < ns ? sd.z - sd.y : 0;
      c_i1 = slice_i1[sl];
      // the descriptors are needed at once; waiting for them here (and for the
      // older loads) leaves nothing of this path pending where it rejoins the
      // in-chunk path, whose waits the compiler would otherwise make as strict
      vm_wait_all();
    }
  };

  // Row-group descriptors, lane P holding group P of a quad (slice j owns
  // ceil(nr_j / GR) consecutive groups): first row | j << 25 | (real rows - 1) << 27,
  // and for D3 = 8 the i3 of both rows; for D3 = 2 the position of the group's first row
  // in the quad's row list (slice 0's rows, then slice 1's, ...: at most 128), whose i3
  // values lanes L and L + 64 hold in d_i3lo / d_i3hi.  Built for the next quad while the
  // current one runs (e_*), then made current (d_*).
  int d_ra = 0, d_ia = 0, d_ib = 0, np = 0;
  int e_ra = 0, e_ia = 0, e_ib = 0, e_np = 0;
  int d_i3lo = 0, d_i3hi = 0, e_i3lo = 0, e_i3hi = 0;
  auto build_desc = [&]() {
    const int n0 = __builtin_amdgcn_readlane(c_nr, qd), n1 = __builtin_amdgcn_readlane(c_nr, qd + 1);
    const int n2 = __builtin_amdgcn_readlane(c_nr, qd + 2), n3 = __builtin_amdgcn_readlane(c_nr, qd + 3);
    const int b0 = __builtin_amdgcn_readlane(c_rb, qd), b1 = __builtin_amdgcn_readlane(c_rb, qd + 1);
    const int b2 = __builtin_amdgcn_readlane(c_rb, qd + 2), b3 = __builtin_amdgcn_readlane(c_rb, qd + 3);
    const int q1 = (n0 + GR - 1) / GR, q2 = q1 + (n1 + GR - 1) / GR, q3 = q2 + (n2 + GR - 1) / GR;
    e_np = q3 + (n3 + GR - 1) / GR;
    // group P of slice j starts at row base_j + GR P and holds min(GR, lim_j - GR P) rows,
    // with the wave-uniform base_j = b_j - GR q_j, lim_j = n_j + GR q_j
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
    const int left = lim - GR * lane;
    const int cnt = ok ? (left < GR ? left : GR) : 1;
    const int ra = ok ? base + GR * lane : b0;  // lanes past the quad's groups keep a valid row
    if (D3 == 8) {
      e_ia = uniq_i3[ra];
      e_ib = uniq_i3[cnt > 1 ? ra + 1 : ra];
    } else {
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
      int pj = 0;
      pj = s1 ? p1 : pj;
      pj = s2 ? p2 : pj;
      pj = s3 ? p3 : pj;
      const int qj = s3 ? q3 : (s2 ? q2 : (s1 ? q1 : 0));
      e_ia = pj + GR * (lane - qj);
    }
    e_ra = ra | (j << 25) | ((cnt - 1) << 27);
  };
  // stage-1 A operand of the quad at qd: Astack[(slice aj, j1 = lane & 3)][a = 4 s + l4]
  // (missing slices repeat the first; their rows are never read)
  float Aop[8];
  auto load_A = [&]() {
    const int nq4 = ns - qd < 4 ? ns - qd : 4;
    const int aj = l15 >> 2;
    const int i1a = __builtin_amdgcn_readlane(c_i1, qd), i1b = __builtin_amdgcn_readlane(c_i1, qd + 1);
    const int i1c = __builtin_amdgcn_readlane(c_i1, qd + 2), i1d = __builtin_amdgcn_readlane(c_i1, qd + 3);
    const float* Ag = G1 + (uint32_t)(t * s.n1 + sel4(aj < nq4 ? aj : 0, i1a, i1b, i1c, i1d)) * 128u +
                      (uint32_t)((lane & 3) * 32 + l4);
#pragma unroll
    for (int s4 = 0; s4 < 8; ++s4) Aop[s4] = Ag[4 * s4];
  };

  struct FPair {
    float d[8];
    int ra;   // first row of the group (wave-uniform)
    int j;    // slice within the quad (wave-uniform)
    int cnt;  // real rows of the group (wave-uniform)
  };
  buf_t g3buf = make_buf(G3, 0);  // G3[t] of the current quad
  auto pair_load = [&](FPair& X, int P) {
    const int rw = __builtin_amdgcn_readlane(d_ra, P);
    X.ra = rw & 0x01FFFFFF;
    X.j = (rw >> 25) & 3;
    X.cnt = ((rw >> 27) & 7) + 1;
    uint32_t i3;
    if (D3 == 8) {
      const int ia = __builtin_amdgcn_readlane(d_ia, P), ib = __builtin_amdgcn_readlane(d_ib, P);
      i3 = (uint32_t)(asel ? ib : ia);
    } else {
      // i3 of this lane's row of the group (rows past the last real one repeat it), read
      // from the lane of the row list that holds it
      const int x = __builtin_amdgcn_readlane(d_ia, P) + (asel < X.cnt ? asel : X.cnt - 1);
      const int lo = __builtin_amdgcn_ds_bpermute(4 * x, d_i3lo), hi = __builtin_amdgcn_ds_bpermute(4 * x, d_i3hi);
      i3 = (uint32_t)(x < 64 ? lo : hi);
    }
    const uint32_t o = vo_d + i3 * G3ROW;
    if (D3 == 8) {
#pragma unroll
      for (int k = 0; k < 8; ++k) X.d[k] = buf_f32(g3buf, o, 16u * D3 * k);
    } else {
      const float4 lo = buf_f32x4(g3buf, o), hi = buf_f32x4(g3buf, o + 16u);
      X.d[0] = lo.x; X.d[1] = lo.y; X.d[2] = lo.z; X.d[3] = lo.w;
      X.d[4] = hi.x; X.d[5] = hi.y; X.d[6] = hi.z; X.d[7] = hi.w;
    }
  };

  FPair XA, XB;
  // B of the chunk's run: loaded before the quad's first row pairs, since vector
  // memory counts complete in issue order (a B loaded after them would make stage 1
  // wait for the row pairs too)
  auto load_B = [&]() {
    if (run != cur_run) {
      const float* Bg = G2 + (uint32_t)run * 4096u + (uint32_t)(l4 * 128 + l15);
#pragma unroll
      for (int s4 = 0; s4 < 8; ++s4)
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) Bop[8 * s4 + nt] = Bg[s4 * 512 + 16 * nt];
      cur_run = run;
    }
  };
  // Stage 1 of a quad, Cstack (16 x 128) = Astack (16 x 32) . B (32 x 128) with rows
  // (slice, j1) and columns (j2, b), in eight groups of eight MFMAs (one contraction
  // step s4 each), so that the next quad's groups can run between the current quad's
  // row pairs; the result waits in Cs until the current quad's C^T reads are done.
  // Rows of slices beyond the chunk's end come from a repeated slice and are never read.
  f32x4 Cs[8];
  auto s1_zero = [&]() {
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) Cs[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  };
  auto s1_group = [&](int s4) {
#pragma unroll
    for (int nt = 0; nt < 8; ++nt)
      Cs[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(Aop[s4], Bop[8 * s4 + nt], Cs[nt], 0, 0, 0);
  };
  auto s1_store = [&]() {
    // lane holds C[slice l4][j1 r][j2 = nt >> 1][b = 16 (nt & 1) + l15]
#pragma unroll
    for (int nt = 0; nt < 8; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) scr_w[F32_ROW * (4 * r + (nt >> 1)) + 16 * (nt & 1)] = Cs[nt][r];
    wave_lds_sync();
  };
  next_chunk();
  if (c >= 0) {
    build_desc();
    load_A();
    d_ra = e_ra;
    d_ia = e_ia;
    d_ib = e_ib;
    d_i3lo = e_i3lo;
    d_i3hi = e_i3hi;
    np = e_np;
    g3buf = make_buf(G3 + (uint32_t)(t * s.n3) * (G3ROW / 4), (uint32_t)s.n3 * G3ROW);
    load_B();
    pair_load(XA, 0);
    pair_load(XB, np > 1 ? 1 : 0);
    s1_zero();
#pragma unroll
    for (int s4 = 0; s4 < 8; ++s4) s1_group(s4);
    s1_store();
  }
  while (c >= 0) {
    // the next quad (the rest of this chunk, or a new chunk claimed now): its
    // descriptors, stage-1 A operand and (new run) B load while this quad's rows are
    // computed; this quad's B is no longer needed
    if (qd + 4 >= ns)
      next_chunk();
    else
      qd += 4;
    const bool nxt = c >= 0;
    if (nxt) {
      build_desc();
      load_A();
      load_B();
    }
    // stage-2 B operand of slice j: C'^T[b = 4 s + l4][jj = l15]
    float CT[8];
    auto slice_begin = [&](int j) {
#pragma unroll
      for (int s4 = 0; s4 < 8; ++s4) CT[s4] = scr_r[F32_SLICE * j + (D3 == 2 ? 1 : 4) * s4];
    };
    slice_begin(0);
    // E rows of a group through a descriptor that ends after the group's real rows, so
    // the rows past them (padding of a short group) are not written
    auto pair_compute = [&](const FPair& X) {
      float Aw[8];
      if (D3 == 8) {
#pragma unroll
        for (int s4 = 0; s4 < 8; ++s4) Aw[s4] = X.d[s4];
      } else {
        // the even lane holds (b, j3) for b = 8 l4 + 0..3, the odd lane for b = 8 l4 + 4..7,
        // both j3 interleaved; each keeps its own j3 and takes the rest from its neighbour
        // (the swaps run on every lane, outside the selects, so that no lane mask hides a
        // neighbour's value)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float from_even = swap_neighbour(X.d[2 * i + 1]), from_odd = swap_neighbour(X.d[2 * i]);
          Aw[i] = odd_lane ? from_even : X.d[2 * i];
          Aw[4 + i] = odd_lane ? X.d[2 * i + 1] : from_odd;
        }
      }
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s4 = 0; s4 < 8; ++s4) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(Aw[s4], CT[s4], acc, 0, 0, 0);
      const buf_t eb = make_buf(E + (size_t)(uint32_t)X.ra * DW, (uint32_t)X.cnt * (4u * DW));
      if (D3 == 8) {
        // lane holds E[row l4 / 2][jj = l15][j3 = 4 (l4 & 1) + r]
        if (e_nt)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc), eb, vo_e, 0, CPOL_NT);
        else
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc), eb, vo_e, 0, 0);
      } else {
        // lane holds E[row 2 l4 + (r / 2)][jj = l15][j3 = r % 2]
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 e01 = u32x2{__float_as_uint(acc[0]), __float_as_uint(acc[1])};
        const u32x2 e23 = u32x2{__float_as_uint(acc[2]), __float_as_uint(acc[3])};
        if (e_nt) {
          __builtin_amdgcn_raw_buffer_store_b64(e01, eb, vo_e, 0, CPOL_NT);
          __builtin_amdgcn_raw_buffer_store_b64(e23, eb, vo_e + 4u * DW, 0, CPOL_NT);
        } else {
          __builtin_amdgcn_raw_buffer_store_b64(e01, eb, vo_e, 0, 0);
          __builtin_amdgcn_raw_buffer_store_b64(e23, eb, vo_e + 4u * DW, 0, 0);
        }
      }
    };
    int cj = 0;
    auto step = [&](const FPair& X) {
      if (X.j != cj) {
        slice_begin(X.j);
        cj = X.j;
      }
      pair_compute(X);
    };
    // the first eight row pairs (loads past the last pair are clamped repeats), each
    // followed by one stage-1 group of the next quad, then the rest
    if (nxt) s1_zero();
    int P = 0;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      pair_load(XB, P + 1 < np ? P + 1 : np - 1);
      if (P < np) step(XA);
      if (nxt) s1_group(2 * g);
      pair_load(XA, P + 2 < np ? P + 2 : np - 1);
      if (P + 1 < np) step(XB);
      if (nxt) s1_group(2 * g + 1);
      P += 2;
    }
    for (; P < np; P += 2) {
      pair_load(XB, P + 1 < np ? P + 1 : np - 1);
      step(XA);
      pair_load(XA, P + 2 < np ? P + 2 : np - 1);
      if (P + 1 < np) step(XB);
    }
    wave_lds_sync();
    // the next quad becomes current: its C into the tile, its first two row pairs load
    if (nxt) {
      s1_store();
      d_ra = e_ra;
      d_ia = e_ia;
      d_ib = e_ib;
      d_i3lo = e_i3lo;
      d_i3hi = e_i3hi;
      np = e_np;
      g3buf = make_buf(G3 + (uint32_t)(t * s.n3) * (G3ROW / 4), (uint32_t)s.n3 * G3ROW);
      pair_load(XA, 0);
      pair_load(XB, np > 1 ? 1 : 0);
    }
  }
}

// ---------------------------------------------------------------------------
// MFMA forward for d = (4, 4, 8), R = 64 (D = 128).  The chunk, quad and row-pair
// structure of the R = 32 kernel; B = G2[t][i2] (64 x 256 floats) no longer fits in
// registers and streams from L2, two column tiles at a time:
//   * stage 1: Cstack (16 x 256) = Astack (16 x 64) . B (64 x 256), 256 MFMAs per
//     quad, with the contraction index a = 16 (lane >> 4) + s, so a lane's sixteen A
//     values are four 16-byte loads;
//   * Cstack goes to a per-wave LDS tile with rows (slice, j1, j2) of 68 floats, the
//     four slices 1,104 floats apart (the writes of a tile take 64 distinct banks);
//   * stage 2 per row pair: E^T = D^T . C'^T, 16 MFMAs, with b = 16 (lane >> 4) + s,
//     so a lane's sixteen C'^T values are four 16-byte LDS reads.
// ---------------------------------------------------------------------------
constexpr int F64_WAVES = 4;
constexpr int F64_WG_PER_CU = 2;
constexpr int F64_PITCH = 68;
constexpr int F64_SLICE = 16 * F64_PITCH + 16;
constexpr int F64_SCR = 4 * F64_SLICE;

__global__ void __launch_bounds__(64 * F64_WAVES, F64_WG_PER_CU)
    k_fwd_r64(ShapeArgs s, const float* __restrict__ G1, const float* __restrict__ G2, const float* __restrict__ G3,
              const int4* __restrict__ slices, const int32_t* __restrict__ slice_i1,
              const int4* __restrict__ chunks, const uint32_t* __restrict__ run_base,
              const int32_t* __restrict__ uniq_i3, int32_t* __restrict__ ctr, float* __restrict__ E) {
  __shared__ float scr_all[F64_WAVES * F64_SCR];
  const int lane = lane_id();
  // E rows of all unique rows beyond the last-level cache: stored non-temporally
  const bool e_nt = (uint64_t)(uint32_t)ctr[C_U] * 512u > STREAM_BYTES;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float* scr = scr_all + wave * F64_SCR;
  const int nch = (int)run_base[s.T * s.n2];
  const int l15 = lane & 15, l4 = lane >> 4;
  const int orow = l4 >> 1;
  const int asel = l15 >> 3;
  // byte offsets: stage-2 A word D^T[(sel, j3 = l15 & 7)][b = 16 l4 + s] in a G3 row
  // (+ 32 bytes per s), the E store (as for R = 32), and the stage-1 B word
  // B[a = 16 l4 + s][16 nt + l15] in G2[t][i2] (+ 1,024 bytes per s, + 64 per nt)
  const uint32_t vo_d = 4u * (uint32_t)(l4 * 128 + (l15 & 7));
  const uint32_t vo_e = 4u * (uint32_t)(orow * 128 + l15 * 8 + 4 * (l4 & 1));
  const uint32_t vo_b = 4u * (uint32_t)(l4 * 4096 + l15);
  // stage-1 output word (slice l4, j1 r, j2, b) and stage-2 operand read (slice j, jj = l15, b = 16 l4 + 4 q)
  const int wr_base = l4 * F64_SLICE + l15;
  const int rd_base = l15 * F64_PITCH + 16 * l4;

  int cursor = 0;
  int c_rb = 0, c_nr = 0, c_i1 = 0;
  int f = 0, ns = 0, run = -1, t = 0, qd = 0;
  int c = -1;
  const int wid = blockIdx.x * F64_WAVES + wave, nw = gridDim.x * F64_WAVES;
  int st_next = share_lo(nch, nw, wid);
  const int st_hi = share_lo(nch, nw, wid + 1);
  auto next_chunk = [&]() {
    if (sched_static(s.sched))
      c = st_next < st_hi ? st_next++ : -1;
    else
      c = claim_queues(ctr + C_FWD_CTR, nch, SCHED_NQ, blockIdx.x % SCHED_NQ, &cursor);
    qd = 0;
    if (c >= 0) {
      const int4 ch = chunks[c];
      f = __builtin_amdgcn_readfirstlane(ch.x);
      ns = __builtin_amdgcn_readfirstlane(ch.y);
      run = __builtin_amdgcn_readfirstlane(ch.z);
      t = run / s.n2;
      const int sl = f + (lane < ns ? lane : 0);
      const int4 sd = slices[sl];
      c_rb = sd.y;
      c_nr = lane < ns ? sd.z - sd.y : 0;
      c_i1 = slice_i1[sl];
    }
  };

  int d_ra = 0, d_ia = 0, d_ib = 0, np = 0;
  int e_ra = 0, e_ia = 0, e_ib = 0, e_np = 0;
  auto build_desc = [&]() {
    const int n0 = __builtin_amdgcn_readlane(c_nr, qd), n1 = __builtin_amdgcn_readlane(c_nr, qd + 1);
    const int n2 = __builtin_amdgcn_readlane(c_nr, qd + 2), n3 = __builtin_amdgcn_readlane(c_nr, qd + 3);
    const int b0 = __builtin_amdgcn_readlane(c_rb, qd), b1 = __builtin_amdgcn_readlane(c_rb, qd + 1);
    const int b2 = __builtin_amdgcn_readlane(c_rb, qd + 2), b3 = __builtin_amdgcn_readlane(c_rb, qd + 3);
    const int q1 = (n0 + 1) >> 1, q2 = q1 + ((n1 + 1) >> 1), q3 = q2 + ((n2 + 1) >> 1);
    e_np = q3 + ((n3 + 1) >> 1);
    // pair P of slice j starts at row base_j + 2 P and has a second row iff
    // 2 P + 1 < lim_j, with the wave-uniform base_j = b_j - 2 q_j, lim_j = n_j + 2 q_j
    const bool s1 = lane >= q1, s2 = lane >= q2, s3 = lane >= q3;
    const int j = (int)s1 + (int)s2 + (int)s3;
    int base = b0, lim = n0;
    base = s1 ? b1 - 2 * q1 : base;
    lim = s1 ? n1 + 2 * q1 : lim;
    base = s2 ? b2 - 2 * q2 : base;
    lim = s2 ? n2 + 2 * q2 : lim;
    base = s3 ? b3 - 2 * q3 : base;
    lim = s3 ? n3 + 2 * q3 : lim;
    const bool ok = lane < e_np;
    const bool has1 = ok && 2 * lane + 1 < lim;
    const int ra = ok ? base + 2 * lane : b0;
    e_ia = uniq_i3[ra];
    e_ib = uniq_i3[has1 ? ra + 1 : ra];
    e_ra = ra | (j << 28) | (has1 ? 1 << 30 : 0);
  };
  // stage-1 A operand of the quad at qd: Astack[(slice aj, j1 = lane & 3)][a = 16 l4 + s]
  float4 A4[4];
  auto load_A = [&]() {
    const int nq4 = ns - qd < 4 ? ns - qd : 4;
    const int aj = l15 >> 2;
    const int i1a = __builtin_amdgcn_readlane(c_i1, qd), i1b = __builtin_amdgcn_readlane(c_i1, qd + 1);
    const int i1c = __builtin_amdgcn_readlane(c_i1, qd + 2), i1d = __builtin_amdgcn_readlane(c_i1, qd + 3);
    const float4* Ag = reinterpret_cast<const float4*>(
        G1 + (uint32_t)(t * s.n1 + sel4(aj < nq4 ? aj : 0, i1a, i1b, i1c, i1d)) * 256u +
        (uint32_t)((lane & 3) * 64 + 16 * l4));
#pragma unroll
    for (int q = 0; q < 4; ++q) A4[q] = Ag[q];
  };

  struct FPair {
    float d[16];
    int ra;
    int j;
    bool has1;
  };
  buf_t g3buf = make_buf(G3, 0);
  auto pair_load = [&](FPair& X, int P) {
    const int rw = __builtin_amdgcn_readlane(d_ra, P);
    const int ia = __builtin_amdgcn_readlane(d_ia, P), ib = __builtin_amdgcn_readlane(d_ib, P);
    X.ra = rw & 0x0FFFFFFF;
    X.j = (rw >> 28) & 3;
    X.has1 = (rw >> 30) & 1;
    const uint32_t o = vo_d + (uint32_t)(asel ? ib : ia) * 2048u;
#pragma unroll
    for (int k = 0; k < 16; ++k) X.d[k] = buf_f32(g3buf, o + 32u * k);
  };

  FPair XA, XB;
  next_chunk();
  if (c >= 0) {
    build_desc();
    load_A();
    d_ra = e_ra;
    d_ia = e_ia;
    d_ib = e_ib;
    np = e_np;
    g3buf = make_buf(G3 + (uint32_t)(t * s.n3) * 512u, (uint32_t)s.n3 * 2048u);
    pair_load(XA, 0);
    pair_load(XB, np > 1 ? 1 : 0);
  }
  while (c >= 0) {
    // stage 1, two column tiles at a time (rows of slices beyond the chunk's end
    // come from a repeated slice and are never read)
    {
      const buf_t bbuf = make_buf(G2 + (uint32_t)run * 16384u, 65536u);
      float Aop[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        Aop[4 * q + 0] = A4[q].x;
        Aop[4 * q + 1] = A4[q].y;
        Aop[4 * q + 2] = A4[q].z;
        Aop[4 * q + 3] = A4[q].w;
      }
#pragma unroll
      for (int p2 = 0; p2 < 8; ++p2) {
        float b0[16], b1[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          b0[k] = buf_f32(bbuf, vo_b + 128u * p2, 1024u * k);
          b1[k] = buf_f32(bbuf, vo_b + 128u * p2 + 64u, 1024u * k);
        }
        f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          c0 = __builtin_amdgcn_mfma_f32_16x16x4f32(Aop[k], b0[k], c0, 0, 0, 0);
          c1 = __builtin_amdgcn_mfma_f32_16x16x4f32(Aop[k], b1[k], c1, 0, 0, 0);
        }
        // lane holds C[slice l4][j1 r][j2 = nt >> 2][b = 16 (nt & 3) + l15], nt = 2 p2 (+1)
        const int nt0 = 2 * p2, nt1 = 2 * p2 + 1;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          scr[wr_base + (4 * r + (nt0 >> 2)) * F64_PITCH + 16 * (nt0 & 3)] = c0[r];
          scr[wr_base + (4 * r + (nt1 >> 2)) * F64_PITCH + 16 * (nt1 & 3)] = c1[r];
        }
      }
      wave_lds_sync();
    }
    if (qd + 4 >= ns)
      next_chunk();
    else
      qd += 4;
    if (c >= 0) {
      build_desc();
      load_A();
    }
    // stage-2 B operand of slice j: C'^T[b = 16 l4 + s][jj = l15]
    float CT[16];
    auto slice_begin = [&](int j) {
      const float4* rp = reinterpret_cast<const float4*>(scr + j * F64_SLICE + rd_base);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = rp[q];
        CT[4 * q + 0] = v.x;
        CT[4 * q + 1] = v.y;
        CT[4 * q + 2] = v.z;
        CT[4 * q + 3] = v.w;
      }
    };
    slice_begin(0);
    auto pair_compute = [&](const FPair& X) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < 16; ++k) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(X.d[k], CT[k], acc, 0, 0, 0);
      const buf_t eb = make_buf(E + (size_t)(uint32_t)X.ra * 128, X.has1 ? 1024u : 512u);
      if (e_nt)
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc), eb, vo_e, 0, CPOL_NT);
      else
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc), eb, vo_e, 0, 0);
    };
    int cj = 0;
    auto step = [&](const FPair& X) {
      if (X.j != cj) {
        slice_begin(X.j);
        cj = X.j;
      }
      pair_compute(X);
    };
    for (int P = 0; P < np; P += 2) {
      pair_load(XB, P + 1 < np ? P + 1 : np - 1);
      step(XA);
      pair_load(XA, P + 2 < np ? P + 2 : np - 1);
      if (P + 1 < np) step(XB);
    }
    wave_lds_sync();
    if (c >= 0) {
      d_ra = e_ra;
      d_ia = e_ia;
      d_ib = e_ib;
      np = e_np;
      g3buf = make_buf(G3 + (uint32_t)(t * s.n3) * 512u, (uint32_t)s.n3 * 2048u);
      pair_load(XA, 0);
      pair_load(XB, np > 1 ? 1 : 0);
    }
  }
}

// Sum pooling: LPB lanes per bag, float4 columns, occurrences in position order.
template <int LPB>
__global__ void __launch_bounds__(256) k_pool4(const float4* __restrict__ E, const int32_t* __restrict__ inv,
                                               const int64_t* __restrict__ offsets, int64_t M, int64_t NB, int D4,
                                               float4* __restrict__ out) {
  const int64_t gb = (int64_t)blockIdx.x * (256 / LPB) + threadIdx.x / LPB;
  const int sub = threadIdx.x % LPB;
  if (gb >= NB) return;
  int64_t lo, hi;
  if (offsets) {
    lo = offsets[gb];
    hi = offsets[gb + 1];
    lo = lo < 0 ? 0 : (lo > M ? M : lo);
    hi = hi < lo ? lo : (hi > M ? M : hi);
  } else {
    lo = gb;
    hi = gb + 1;
  }
  for (int j = sub; j < D4; j += LPB) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    int64_t o = lo;
    for (; o + 4 <= hi; o += 4) {
      const int u0 = inv[o], u1 = inv[o + 1], u2 = inv[o + 2], u3 = inv[o + 3];
      float4 e0 = u0 >= 0 ? E[(int64_t)u0 * D4 + j] : make_float4(0.f, 0.f, 0.f, 0.f);
      float4 e1 = u1 >= 0 ? E[(int64_t)u1 * D4 + j] : make_float4(0.f, 0.f, 0.f, 0.f);
      float4 e2 = u2 >= 0 ? E[(int64_t)u2 * D4 + j] : make_float4(0.f, 0.f, 0.f, 0.f);
      float4 e3 = u3 >= 0 ? E[(int64_t)u3 * D4 + j] : make_float4(0.f, 0.f, 0.f, 0.f);
      acc.x += e0.x; acc.y += e0.y; acc.z += e0.z; acc.w += e0.w;
      acc.x += e1.x; acc.y += e1.y; acc.z += e1.z; acc.w += e1.w;
      acc.x += e2.x; acc.y += e2.y; acc.z += e2.z; acc.w += e2.w;
      acc.x += e3.x; acc.y += e3.y; acc.z += e3.z; acc.w += e3.w;
    }
    for (; o < hi; ++o) {
      const int u = inv[o];
      if (u >= 0) {
        float4 e = E[(int64_t)u * D4 + j];
        acc.x += e.x; acc.y += e.y; acc.z += e.z; acc.w += e.w;
      }
    }
    out[gb * D4 + j] = acc;
  }
}

// D = 128: two bags per wave, 32 lanes and one float4 column each.  Each half
// reads up to 32 of its bag's row indices in one load; 16 rows per half are in
// flight before they are summed in occurrence order.
__global__ void __launch_bounds__(256) k_pool128(const float4* __restrict__ E, const int32_t* __restrict__ inv,
                                                 const int64_t* __restrict__ offsets, int64_t M, int64_t NB,
                                                 float4* __restrict__ out) {
  const int lane = lane_id();
  const int half = lane >> 5, sub = lane & 31;
  const int64_t gb = ((int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6)) * 2 + half;
  const bool bag_ok = gb < NB;
  int64_t lo = 0, hi = 0;
  if (bag_ok) {
    if (offsets) {
      lo = offsets[gb];
      hi = offsets[gb + 1];
      lo = lo < 0 ? 0 : (lo > M ? M : lo);
      hi = hi < lo ? lo : (hi > M ? M : hi);
    } else {
      lo = gb;
      hi = gb + 1;
    }
  }
  const int cnt = (int)(hi - lo);
  const int c0 = __builtin_amdgcn_readlane(cnt, 0), c1 = __builtin_amdgcn_readlane(cnt, 32);
  const int cmax = c0 > c1 ? c0 : c1;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int base = 0; base < cmax; base += 32) {
    const int my_u = base + sub < cnt ? inv[lo + base + sub] : -1;
    const int nb = cmax - base < 32 ? cmax - base : 32;
    for (int k0 = 0; k0 < nb; k0 += 16) {
      float4 v[16];
#pragma unroll
      for (int kk = 0; kk < 16; ++kk) {
        const int k = k0 + kk;
        const int uA = __builtin_amdgcn_readlane(my_u, k & 31), uB = __builtin_amdgcn_readlane(my_u, 32 + (k & 31));
        const int u = half ? uB : uA;
        if (base + k < cnt) v[kk] = E[(size_t)(u < 0 ? 0 : u) * 32 + sub];  // invalid rows: row 0, skipped
      }
#pragma unroll
      for (int kk = 0; kk < 16; ++kk) {
        const int k = k0 + kk;
        const int uA = __builtin_amdgcn_readlane(my_u, k & 31), uB = __builtin_amdgcn_readlane(my_u, 32 + (k & 31));
        const int u = half ? uB : uA;
        if (base + k < cnt && u >= 0) {
          acc.x += v[kk].x;
          acc.y += v[kk].y;
          acc.z += v[kk].z;
          acc.w += v[kk].w;
        }
      }
    }
  }
  if (bag_ok) out[gb * 32 + sub] = acc;
}

__global__ void __launch_bounds__(256) k_pool1(const float* __restrict__ E, const int32_t* __restrict__ inv,
                                               const int64_t* __restrict__ offsets, int64_t M, int64_t NB, int D,
                                               float* __restrict__ out) {
  const int64_t gb = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (gb >= NB) return;
  int64_t lo, hi;
  if (offsets) {
    lo = offsets[gb];
    hi = offsets[gb + 1];
    lo = lo < 0 ? 0 : (lo > M ? M : lo);
    hi = hi < lo ? lo : (hi > M ? M : hi);
  } else {
    lo = gb;
    hi = gb + 1;
  }
  for (int j = lane_id(); j < D; j += 64) {
    float acc = 0.f;
    for (int64_t o = lo; o < hi; ++o) {
      const int u = inv[o];
      if (u >= 0) acc += E[(int64_t)u * D + j];
    }
    out[gb * D + j] = acc;
  }
}

int persistent_grid() {
  static int cached = 0;
  if (!cached) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
      cached = cus;
    else
      cached = 256;
  }
  return cached;
}

hipError_t launch_pool(const Shape& s, const float* E, const int32_t* inv, const int64_t* offsets, int64_t M,
                       int64_t B, float* out, const Prof& prof, hipStream_t st) {
  const int64_t NB = (int64_t)s.T * B;
  if (NB <= 0) return hipSuccess;
  prof_begin(prof, K_POOL, st);
  if (s.D == 128) {
    hipLaunchKernelGGL(k_pool128, dim3((unsigned)((NB + 7) / 8)), dim3(256), 0, st,
                       reinterpret_cast<const float4*>(E), inv, offsets, M, NB, reinterpret_cast<float4*>(out));
  } else if (s.D % 4 == 0) {
    const int D4 = s.D / 4;
    int lpb = 1;
    while (lpb < D4 && lpb < 64) lpb <<= 1;
    const int64_t per = 256 / lpb;
    const dim3 grid((unsigned)((NB + per - 1) / per));
    const float4* E4 = reinterpret_cast<const float4*>(E);
    float4* o4 = reinterpret_cast<float4*>(out);
    switch (lpb) {
      case 1: hipLaunchKernelGGL(k_pool4<1>, grid, dim3(256), 0, st, E4, inv, offsets, M, NB, D4, o4); break;
      case 2: hipLaunchKernelGGL(k_pool4<2>, grid, dim3(256), 0, st, E4, inv, offsets, M, NB, D4, o4); break;
      case 4: hipLaunchKernelGGL(k_pool4<4>, grid, dim3(256), 0, st, E4, inv, offsets, M, NB, D4, o4); break;
      case 8: hipLaunchKernelGGL(k_pool4<8>, grid, dim3(256), 0, st, E4, inv, offsets, M, NB, D4, o4); break;
      case 16: hipLaunchKernelGGL(k_pool4<16>, grid, dim3(256), 0, st, E4, inv, offsets, M, NB, D4, o4); break;
      case 32: hipLaunchKernelGGL(k_pool4<32>, grid, dim3(256), 0, st, E4, inv, offsets, M, NB, D4, o4); break;
      default: hipLaunchKernelGGL(k_pool4<64>, grid, dim3(256), 0, st, E4, inv, offsets, M, NB, D4, o4); break;
    }
  } else {
    hipLaunchKernelGGL(k_pool1, dim3((unsigned)((NB + 3) / 4)), dim3(256), 0, st, E, inv, offsets, M, NB, s.D, out);
  }
  prof_end(prof, K_POOL, st);
  return hipGetLastError();
}

bool fwd_r64_supported(const Shape& s, int64_t max_indices) {
  // 32-bit offsets into E (rows x 128), G1, G2 and G3; a table's G3 (n3 x 2,048 bytes) is
  // one buffer descriptor's 32-bit range
  return s.d1 == 4 && s.d2 == 4 && s.d3 == 8 && s.R == 64 && max_indices * 128 < (int64_t(1) << 31) &&
         (int64_t)s.T * s.n1 * 256 < (int64_t(1) << 31) && (int64_t)s.T * s.n2 * 16384 < (int64_t(1) << 31) &&
         (int64_t)s.T * s.n3 * 512 < (int64_t(1) << 31) && (int64_t)s.n3 * 2048 < (int64_t(1) << 32);
}

bool fwd_r32_supported(const Shape& s, int64_t max_indices) {
  // d = (4, 4, 8) or (4, 4, 2); 32-bit float offsets into E (rows x at most 128), G1 (slices of 128),
  // G2 (slices of 4,096) and G3 (slices of at most 256) must fit (so do the 25-bit rows of a descriptor)
  return s.d1 == 4 && s.d2 == 4 && (s.d3 == 8 || s.d3 == 2) && s.R == 32 && max_indices * 128 < (int64_t(1) << 31) &&
         (int64_t)s.T * s.n3 * 256 < (int64_t(1) << 31) && (int64_t)s.T * s.n1 * 128 < (int64_t(1) << 31) &&
         (int64_t)s.T * s.n2 * 4096 < (int64_t(1) << 31);
}

hipError_t launch_forward(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                          const int64_t* offsets, int64_t M, int64_t B, float* out, const Prof& prof,
                          hipStream_t st) {
  if (M > 0) {
    const int grid = persistent_grid() * 2;
    hipError_t e = fill_u32(reinterpret_cast<uint32_t*>(w.ctr + C_FWD_CTR), SCHED_NQ * SCHED_STRIDE, 0u, st);
    if (e != hipSuccess) return e;
    if (fwd_r32_supported(s, M)) {
      const int blocks = persistent_grid() * F32_WG_PER_CU;
      prof_begin(prof, K_FWD_FUSED, st);
      hipLaunchKernelGGL(s.d3 == 8 ? k_fwd_r32<8> : k_fwd_r32<2>, dim3(blocks), dim3(64 * F32_WAVES), 0, st,
                         shape_args(s), G1, G2, G3,
                         (const int4*)w.slices, (const int32_t*)w.slice_i1, (const int4*)w.chunks,
                         (const uint32_t*)w.run_nch, (const int32_t*)w.uniq_i3, w.ctr, w.E);
      prof_end(prof, K_FWD_FUSED, st);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      return launch_pool(s, w.E, w.inv, offsets, M, B, out, prof, st);
    }
    if (fwd_r64_supported(s, M)) {
      const int blocks = persistent_grid() * F64_WG_PER_CU;
      prof_begin(prof, K_FWD_FUSED, st);
      hipLaunchKernelGGL(k_fwd_r64, dim3(blocks), dim3(64 * F64_WAVES), 0, st, shape_args(s), G1, G2, G3,
                         (const int4*)w.slices, (const int32_t*)w.slice_i1, (const int4*)w.chunks,
                         (const uint32_t*)w.run_nch, (const int32_t*)w.uniq_i3, w.ctr, w.E);
      prof_end(prof, K_FWD_FUSED, st);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      return launch_pool(s, w.E, w.inv, offsets, M, B, out, prof, st);
    }
    const size_t nC = (size_t)s.d1 * s.d2 * s.R, nA = (size_t)s.d1 * s.R;
    const size_t bs = (size_t)s.R * (s.d2 * s.R + 1);
    const int stage_b = nC + nA + bs <= (size_t)FWD_LDS_FLOATS;
    const size_t lds = sizeof(float) * (nC + nA + (stage_b ? bs : 0));
    const bool wide = nC >= 1024 || s.D >= 128;
    const void* kfn = wide ? (const void*)k_fwd_generic<1024> : (const void*)k_fwd_generic<256>;
    e = hipFuncSetAttribute(kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    if (s.sched == SCHED_STEAL_CKPT) {  // checkpoints of earlier calls may hold other cores' C
      if (!w.ckpt_tag) return hipErrorInvalidValue;
      e = fill_u32(reinterpret_cast<uint32_t*>(w.ckpt_tag), CKPT_SLOTS, (uint32_t)CKPT_EMPTY, st);
      if (e != hipSuccess) return e;
    }
    prof_begin(prof, K_FWD_FUSED, st);
    if (wide)
      hipLaunchKernelGGL(k_fwd_generic<1024>, dim3(grid), dim3(1024), lds, st, shape_args(s), G1, G2, G3,
                         (const int4*)w.slices, (const int4*)w.chunks, (const uint32_t*)w.run_nch,
                         (const int32_t*)w.uniq_i3, w.ctr, w.E, w.ckpt, w.ckpt_tag, stage_b);
    else
      hipLaunchKernelGGL(k_fwd_generic<256>, dim3(grid), dim3(256), lds, st, shape_args(s), G1, G2, G3,
                         (const int4*)w.slices, (const int4*)w.chunks, (const uint32_t*)w.run_nch,
                         (const int32_t*)w.uniq_i3, w.ctr, w.E, w.ckpt, w.ckpt_tag, stage_b);
    prof_end(prof, K_FWD_FUSED, st);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return launch_pool(s, w.E, w.inv, offsets, M, B, out, prof, st);
}

}  // namespace ttemb
