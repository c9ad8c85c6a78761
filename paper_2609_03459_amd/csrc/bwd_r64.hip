// Backward pass for d = (4, 4, 8), R = 64 (D = 128) on MFMA (FlowTT Section 3.2, Eq. 1).
//
// At rank 64 one table's dG3 (n3 x 64 x 8 floats) does not fit in LDS, so this
// kernel keeps no on-chip accumulator.  A wave takes a chunk (consecutive
// slices of one (t, i2) run), four slices ("a quad") at a time:
//   stage 1  Cstack (16 x 256) = Astack (16 x 64) . B (64 x 256), B streamed from
//            L2 (as in the R = 64 forward), into the wave's LDS tile, rows
//            (slice, j1, j2) of 64 columns b;
//   per row pair of slice j:
//            dD^T (16 x 64) = dE^T . C_j   -> the two rows' dD partials, each row's
//                                            512 floats [b][j3] stored contiguously
//            dC_j += dE . D^T              (16 x 64, summed over the slice's rows);
//   slice end: dC_j replaces C_j in the tile (same rows) and goes to the slice's
//              dC partial (d1 x d2 R);
//   quad end:  dA (16 x 64) = dCstack (16 x 256) . B^T  -> per-slice dA partials.
// dB of a (t, i2) run, the sum over its slices of A_s^T dC_s, is formed afterwards
// from the dC partials by k_dg2_r64, one matrix-core product per run with the
// contraction over (slice, j1): a 4 KB partial per slice instead of a 64 KB dB
// partial per chunk.  The fixed-order segment sums of the generic path turn the
// dA and dD partials into dG1 and dG3 (or apply the fused update).
#include "common.h"

namespace ttemb {

ShapeArgs shape_args(const Shape& s);

constexpr int B64_WAVES = 4;
constexpr int B64_WG_PER_CU = 2;
constexpr int B64_PITCH = 68;                     // floats per tile row (64 + pad)
constexpr int B64_SLICE = 16 * B64_PITCH + 16;    // floats per slice in the tile
constexpr int B64_SCR = 4 * B64_SLICE;            // per-wave tile

__global__ void __launch_bounds__(64 * B64_WAVES, B64_WG_PER_CU)
    k_bwd_r64(ShapeArgs s, const float* __restrict__ G1, const float* __restrict__ G2, const float* __restrict__ G3,
              const float* __restrict__ dE, const int4* __restrict__ slices, const int32_t* __restrict__ slice_i1,
              const int4* __restrict__ chunks, const uint32_t* __restrict__ run_base,
              const int32_t* __restrict__ uniq_i3, int32_t* __restrict__ ctr, float* __restrict__ dApart,
              float* __restrict__ dCpart, float* __restrict__ dDpart) {
  __shared__ float scr_all[B64_WAVES * B64_SCR];
  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float* scr = scr_all + wave * B64_SCR;
  const int nch = (int)run_base[s.T * s.n2];
  const int l15 = lane & 15, l4 = lane >> 4;
  // per-row dD partials (2 KB per unique row) beyond the last-level cache: stored
  // non-temporally
  const bool dd_nt = (uint64_t)(uint32_t)ctr[C_U] * 2048u > STREAM_BYTES;
  // byte offsets of this lane's operand words:
  //   stage 1 B[a = 16 l4 + k][16 nt + l15] in G2[t][i2] (+ 1,024 bytes per k, + 64 per nt)
  const uint32_t vo_b = 4u * (uint32_t)(l4 * 4096 + l15);
  //   dE^T[(row, j3) = l15][jj = 4 s + l4] in a pair's two rows (+ 128 bytes per s)
  const uint32_t vo_eb = 4u * (uint32_t)((l15 >> 3) * 128 + l4 * 8 + (l15 & 7));
  //   dE[row = l4 >> 1][jj = l15][j3 = 4 (l4 & 1) + s], s = 0..3: one 16-byte word
  const uint32_t vo_e4 = 4u * (uint32_t)((l4 >> 1) * 128 + l15 * 8 + 4 * (l4 & 1));
  //   G3[i3][b = 16 nt + l15][j3 = 4 (l4 & 1) + s] (+ 512 bytes per nt): one 16-byte word
  const uint32_t vo_d4 = 4u * (uint32_t)(l15 * 8 + 4 * (l4 & 1));
  //   dD partial of row (l4 >> 1), [b = 16 nt + l15][j3 = 4 (l4 & 1) + r] (+ 512 bytes per nt)
  const uint32_t vo_dd = 4u * (uint32_t)((l4 >> 1) * 512 + l15 * 8 + 4 * (l4 & 1));
  // LDS tile: stage-1 write of (slice l4, row 4 r + j2, column b = 16 (nt & 3) + l15)
  const int wr_base = l4 * B64_SLICE + l15;

  int cursor = 0;
  const int wid = blockIdx.x * B64_WAVES + wave, nw = gridDim.x * B64_WAVES;
  int st_next = share_lo(nch, nw, wid);
  const int st_hi = share_lo(nch, nw, wid + 1);
  while (true) {
    int c;
    if (sched_static(s.sched))
      c = st_next < st_hi ? st_next++ : -1;
    else
      c = claim_queues(ctr + C_BWD_CTR, nch, SCHED_NQ, blockIdx.x % SCHED_NQ, &cursor);
    if (c < 0) break;
    const int4 ch = chunks[c];
    const int f = __builtin_amdgcn_readfirstlane(ch.x);
    const int ns = __builtin_amdgcn_readfirstlane(ch.y);
    const int run = __builtin_amdgcn_readfirstlane(ch.z);
    const int t = run / s.n2;
    // slice descriptors, lane j holding slice f + j (j < ns <= 64)
    const int sl = f + (lane < ns ? lane : 0);
    const int4 sd = slices[sl];
    const int c_rb = sd.y, c_nr = lane < ns ? sd.z - sd.y : 0, c_i1 = slice_i1[sl];
    const buf_t bbuf = make_buf(G2 + (size_t)run * 16384, 65536u);
    const buf_t g3buf = make_buf(G3 + (size_t)t * s.n3 * 512, (uint32_t)s.n3 * 2048u);
    for (int qd = 0; qd < ns; qd += 4) {
      const int nqs = ns - qd < 4 ? ns - qd : 4;
      // ---- stage 1: C of the quad's slices (missing slices repeat the first) ----
      {
        const int aj = l15 >> 2;
        const int i1a = __builtin_amdgcn_readlane(c_i1, qd), i1b = __builtin_amdgcn_readlane(c_i1, qd + 1);
        const int i1c = __builtin_amdgcn_readlane(c_i1, qd + 2), i1d = __builtin_amdgcn_readlane(c_i1, qd + 3);
        const float4* Ag = reinterpret_cast<const float4*>(
            G1 + ((size_t)t * s.n1 + sel4(aj < nqs ? aj : 0, i1a, i1b, i1c, i1d)) * 256 + (lane & 3) * 64 + 16 * l4);
        float Aop[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 v = Ag[q];
          Aop[4 * q + 0] = v.x;
          Aop[4 * q + 1] = v.y;
          Aop[4 * q + 2] = v.z;
          Aop[4 * q + 3] = v.w;
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
            scr[wr_base + (4 * r + (nt0 >> 2)) * B64_PITCH + 16 * (nt0 & 3)] = c0[r];
            scr[wr_base + (4 * r + (nt1 >> 2)) * B64_PITCH + 16 * (nt1 & 3)] = c1[r];
          }
        }
        wave_lds_sync();
      }
      // ---- per slice: row pairs, then dC in place of C ----
      for (int j = 0; j < nqs; ++j) {
        const int rb = __builtin_amdgcn_readlane(c_rb, qd + j), nr = __builtin_amdgcn_readlane(c_nr, qd + j);
        // C_j as the dD^T B operand: C[jj = 4 s + l4][b = 16 nt + l15], (nt, s) -> 4 nt + s
        float CB[16];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
          for (int s4 = 0; s4 < 4; ++s4) CB[4 * nt + s4] = scr[j * B64_SLICE + (4 * s4 + l4) * B64_PITCH + 16 * nt + l15];
        f32x4 dC[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) dC[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int r0 = rb; r0 < rb + nr; r0 += 2) {
          const bool has1 = r0 + 1 < rb + nr;
          // rows r0 and r0 + 1 through descriptors that end after the rows that exist:
          // the missing partner of a lone row reads zeros and is not stored
          const buf_t eb = make_buf(dE + (size_t)r0 * 128, has1 ? 1024u : 512u);
          float e_b[4];
#pragma unroll
          for (int s4 = 0; s4 < 4; ++s4) e_b[s4] = buf_f32(eb, vo_eb, 128u * s4);
          const float4 e4 = buf_f32x4(eb, vo_e4);
          const int i3a = uniq_i3[r0];
          const int i3b = has1 ? uniq_i3[r0 + 1] : i3a;
          const uint32_t dbase = (uint32_t)((l4 >> 1) ? i3b : i3a) * 2048u + vo_d4;
          float4 d4[4];
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) d4[nt] = buf_f32x4(g3buf, dbase + 512u * nt);
          const buf_t db = make_buf(dDpart + (size_t)r0 * 512, has1 ? 4096u : 2048u);
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) {
            f32x4 dd = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) dd = __builtin_amdgcn_mfma_f32_16x16x4f32(e_b[s4], CB[4 * nt + s4], dd, 0, 0, 0);
            // lane holds dD[row l4 >> 1][b = 16 nt + l15][j3 = 4 (l4 & 1) + r]
            if (dd_nt)
              __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, dd), db, vo_dd + 512u * nt, 0, CPOL_NT);
            else
              __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, dd), db, vo_dd + 512u * nt, 0, 0);
            dC[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(e4.x, d4[nt].x, dC[nt], 0, 0, 0);
            dC[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(e4.y, d4[nt].y, dC[nt], 0, 0, 0);
            dC[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(e4.z, d4[nt].z, dC[nt], 0, 0, 0);
            dC[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(e4.w, d4[nt].w, dC[nt], 0, 0, 0);
          }
        }
        // lane holds dC[jj = 4 l4 + r][b = 16 nt + l15]: rows of slice j, in place of C_j,
        // and the slice's partial [j1][(j2, b)] = [jj][b]
        wave_lds_sync();
        // the slice's partial, read once by the dG2 product: stored non-temporally
        float* dcs = dCpart + (size_t)(f + qd + j) * 1024 + 4 * l4 * 64 + l15;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            scr[j * B64_SLICE + (4 * l4 + r) * B64_PITCH + 16 * nt + l15] = dC[nt][r];
            __builtin_nontemporal_store(dC[nt][r], dcs + r * 64 + 16 * nt);
          }
      }
      wave_lds_sync();
      // ---- dA (16 x 64) = dCstack (16 x 256) . B^T, contraction (j2, b = 16 l4 + q) ----
      {
        f32x4 acc[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        const float* arow = scr + (l15 >> 2) * B64_SLICE + (l15 & 3) * 4 * B64_PITCH + 16 * l4;
#pragma unroll
        for (int j2 = 0; j2 < 4; ++j2) {
          float av[16];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float4 v = *reinterpret_cast<const float4*>(arow + j2 * B64_PITCH + 4 * q);
            av[4 * q + 0] = v.x;
            av[4 * q + 1] = v.y;
            av[4 * q + 2] = v.z;
            av[4 * q + 3] = v.w;
          }
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) {
            // B^T[(j2, b)][a = 16 nt + l15] = B[a][j2 * 64 + b]
            float bv[16];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const float4 v =
                  buf_f32x4(bbuf, 4u * (uint32_t)((16 * nt + l15) * 256 + j2 * 64 + 16 * l4 + 4 * q));
              bv[4 * q + 0] = v.x;
              bv[4 * q + 1] = v.y;
              bv[4 * q + 2] = v.z;
              bv[4 * q + 3] = v.w;
            }
#pragma unroll
            for (int k = 0; k < 16; ++k) acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[k], bv[k], acc[nt], 0, 0, 0);
          }
        }
        // lane holds dA[slice l4][j1 r][a = 16 nt + l15]; read once, by the dG1 sum: stored
        // non-temporally
        if (l4 < nqs) {
          float* dst = dApart + (size_t)(f + qd + l4) * 256 + l15;
#pragma unroll
          for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int r = 0; r < 4; ++r) __builtin_nontemporal_store(acc[nt][r], dst + r * 64 + 16 * nt);
        }
      }
      wave_lds_sync();
    }
  }
}

bool bwd_r64_supported(const Shape& s, int64_t max_indices) {
  // 32-bit offsets into dE (rows of 128 floats) and the cores (slices of 256, 16,384 and 512
  // floats), and a table's G3 within one buffer descriptor, as for the R = 64 forward; the
  // partials are addressed in 64 bits
  return s.d1 == 4 && s.d2 == 4 && s.d3 == 8 && s.R == 64 && max_indices * 128 < (int64_t(1) << 31) &&
         (int64_t)s.T * s.n1 * 256 < (int64_t(1) << 31) && (int64_t)s.T * s.n2 * 16384 < (int64_t(1) << 31) &&
         (int64_t)s.T * s.n3 * 512 < (int64_t(1) << 31) && (int64_t)s.n3 * 2048 < (int64_t(1) << 32);
}

hipError_t launch_bwd_r64(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                          const Prof& prof, hipStream_t st) {
  hipError_t e = fill_u32(reinterpret_cast<uint32_t*>(w.ctr + C_BWD_CTR), SCHED_NQ * SCHED_STRIDE, 0u, st);
  if (e != hipSuccess) return e;
  const int blocks = persistent_grid() * B64_WG_PER_CU;
  prof_begin(prof, K_BWD_FUSED, st);
  hipLaunchKernelGGL(k_bwd_r64, dim3(blocks), dim3(64 * B64_WAVES), 0, st, shape_args(s), G1, G2, G3,
                     (const float*)w.E, (const int4*)w.slices, (const int32_t*)w.slice_i1, (const int4*)w.chunks,
                     (const uint32_t*)w.run_nch, (const int32_t*)w.uniq_i3, w.ctr, w.dApart, w.dCpart, w.dDpart);
  prof_end(prof, K_BWD_FUSED, st);
  return hipGetLastError();
}

// dG2[t][i2] (R x d2 R) = sum over the slices s of run (t, i2), in slice order, of
// A_s^T . dC_s, with A_s = G1[t][i1 of s] (d1 x R) and dC_s the slice's dC partial
// (d1 x d2 R): a matrix-core product whose contraction index is (slice, j1), one MFMA
// step per slice.  One workgroup per run: wave w takes 32 of the 256 columns (j2, b),
// cg = w % 8, as eight 16 x 16 tiles with the 64 rows a, over the half w / 8 of the run's
// slices, and the halves are added in order through LDS, so the result is the same bits
// run to run.  Few accumulators keep a wave near 64 VGPRs, so two workgroups share a
// CU at eight waves per SIMD, and the waves' operand loads overlap each other's products.
// The slices of a run are contiguous (the (t, i2, i1) slot order): from the slot base of
// (t, i2, 0) to that of the next run.  With `update`, dG2 is G2 itself and receives
// G2 - lr sum; G1 must not have been updated yet (the dG1 reduction runs after this).
constexpr int DG2_WAVES = 16;
__global__ void __launch_bounds__(64 * DG2_WAVES, 8) k_dg2_r64(ShapeArgs s, const float* __restrict__ G1,
                                                               const uint32_t* __restrict__ dense_base,
                                                               const int32_t* __restrict__ slice_i1,
                                                               const int32_t* __restrict__ ctr,
                                                               const float* __restrict__ dCpart,
                                                               float* __restrict__ dG2, float lr, bool update) {
  extern __shared__ float red[];  // the second half's sums: [cg][tile, r][lane]
  const int run = blockIdx.x;
  const int t = run / s.n2;
  const int lane = lane_id(), w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l15 = lane & 15, l4 = lane >> 4;
  const int cg = w & 7, ks = w >> 3;
  const int64_t slot0 = (int64_t)run * s.n1;
  const int lo = (int)dense_base[slot0];
  const int hi = run + 1 < s.T * s.n2 ? (int)dense_base[slot0 + s.n1] : ctr[C_NSLICES];
  const int n = hi - lo;
  const int k0 = lo + (int)(((int64_t)n * ks) / 2), k1 = lo + (int)(((int64_t)n * (ks + 1)) / 2);
  f32x4 acc[8];  // tile (mt, nt) -> 2 mt + nt: rows a = 16 mt + .., columns 32 cg + 16 nt + ..
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float* G1t = G1 + (size_t)t * s.n1 * 256;
  // the half's slices 64 at a time, their i1 in the lanes (one load); per slice the
  // operands A^T[a = 16 mt + l15][j1 = l4] and dC[j1 = l4][32 cg + 16 nt + l15]
  for (int base = k0; base < k1; base += 64) {
    const int cnt = k1 - base < 64 ? k1 - base : 64;
    const int my_i1 = slice_i1[base + (lane < cnt ? lane : 0)];
    for (int k = 0; k < cnt; ++k) {
      const int sl = base + k;
      const float* Ar = G1t + (size_t)__builtin_amdgcn_readlane(my_i1, k) * 256 + l4 * 64 + l15;
      const float* Cr = dCpart + (size_t)sl * 1024 + l4 * 256 + cg * 32 + l15;
      float a[4], b[2];
#pragma unroll
      for (int m = 0; m < 4; ++m) a[m] = Ar[16 * m];
#pragma unroll
      for (int q = 0; q < 2; ++q) b[q] = ntl(Cr + 16 * q);
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int q = 0; q < 2; ++q)
          acc[2 * m + q] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[m], b[q], acc[2 * m + q], 0, 0, 0);
    }
  }
  float* rq = red + cg * 2048 + lane;
  if (ks == 1) {
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int r = 0; r < 4; ++r) rq[(4 * k + r) * 64] = acc[k][r];
  }
  __syncthreads();
  if (ks == 0) {
    // lane holds dG2[a = 16 mt + 4 l4 + r][(j2, b) = 32 cg + 16 nt + l15]
    float* out = dG2 + (size_t)run * 16384 + cg * 32 + l15;
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float v = acc[2 * m + q][r] + rq[(4 * (2 * m + q) + r) * 64];
          float* p = out + (16 * m + 4 * l4 + r) * 256 + 16 * q;
          *p = update ? *p - lr * v : v;
        }
  }
}

hipError_t launch_dg2_r64(const Shape& s, const Work& w, const float* G1, float* dG2, float lr, bool update,
                          hipStream_t st) {
  const int lds = (int)sizeof(float) * 8 * 2048;
  hipError_t e = hipFuncSetAttribute((const void*)k_dg2_r64, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_dg2_r64, dim3(s.T * s.n2), dim3(64 * DG2_WAVES), lds, st, shape_args(s), G1,
                     (const uint32_t*)w.dense_base, (const int32_t*)w.slice_i1, (const int32_t*)w.ctr,
                     (const float*)w.dCpart, dG2, lr, update);
  return hipGetLastError();
}

}  // namespace ttemb
