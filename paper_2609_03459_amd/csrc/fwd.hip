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
  return a;
}

constexpr int FWD_THREADS = 256;
constexpr int FWD_CHUNK = 8;  // slices per scheduler chunk

// Generic fused forward for any shape within the library limits (plain VALU).
__global__ void __launch_bounds__(FWD_THREADS) k_fwd_generic(ShapeArgs s, const float* __restrict__ G1,
                                                             const float* __restrict__ G2,
                                                             const float* __restrict__ G3,
                                                             const int4* __restrict__ slices,
                                                             const uint32_t* __restrict__ uniq_key,
                                                             int32_t* __restrict__ ctr, float* __restrict__ E) {
  extern __shared__ float lds[];
  float* C = lds;  // d1 * d2 * R
  __shared__ int s_chunk;
  const int nsl = ctr[C_NSLICES];
  const int nchunks = (nsl + FWD_CHUNK - 1) / FWD_CHUNK;
  const int d2R = s.d2 * s.R;
  const int nC = s.d1 * d2R;
  int victim = 0;
  int cur_pg = -1;
  while (true) {
    int c = claim_chunk(ctr + C_FWD_CTR, ctr + C_FWD_STEAL, nchunks, &victim, &s_chunk);
    if (c < 0) break;
    const int s0 = c * FWD_CHUNK;
    const int s1 = s0 + FWD_CHUNK < nsl ? s0 + FWD_CHUNK : nsl;
    for (int si = s0; si < s1; ++si) {
      const int4 sl = slices[si];
      const int p = sl.x, rb = sl.y, re = sl.z;
      const uint32_t key = (uint32_t)sl.w;
      const int t = key / s.n12, q = key % s.n12;
      const int i1 = q / s.n2, i2 = q % s.n2;
      if (p != cur_pg) {
        // intermediate C = A.B, kept in LDS while rows of this group follow
        __syncthreads();
        const float* A = G1 + ((int64_t)(t * s.n1 + i1) * s.d1) * s.R;
        const float* Bm = G2 + (int64_t)(t * s.n2 + i2) * s.R * d2R;
        for (int o = threadIdx.x; o < nC; o += FWD_THREADS) {
          const int j1 = o / d2R, cc = o % d2R;
          float acc = 0.f;
          for (int a = 0; a < s.R; ++a) acc = fmaf(A[j1 * s.R + a], Bm[a * d2R + cc], acc);
          C[o] = acc;
        }
        __syncthreads();
        cur_pg = p;
      }
      // embedding rows E_u = C . D_u, C viewed as (d1 d2) x R
      const int total = (re - rb) * s.D;
      for (int o = threadIdx.x; o < total; o += FWD_THREADS) {
        const int r = o / s.D, j = o % s.D;
        const int u = rb + r;
        const int i3 = decode_key(uniq_key[u], s.Npad, s.n2, s.n3).i3;
        const int jr = j / s.d3, j3 = j % s.d3;
        const float* Dm = G3 + (int64_t)(t * s.n3 + i3) * s.R * s.d3;
        float acc = 0.f;
        for (int b = 0; b < s.R; ++b) acc = fmaf(C[jr * s.R + b], Dm[b * s.d3 + j3], acc);
        E[(int64_t)u * s.D + j] = acc;
      }
    }
  }
}


// ---------------------------------------------------------------------------
// MFMA forward for d = (4, 4, 8), R = 32 (D = 128).  Every wave is an
// independent worker over chunks of FWD_CHUNK slices:
//   * B = G2[t][i2] (32 x 128) stays in 64 VGPRs while consecutive slices share
//     (t, i2) (lane l holds columns l and l + 64 of every row k);
//   * stage 1, C = A.B (4 x 128), per prefix group with v_mfma_f32_4x4x1f32
//     (16 blocks of 4x4; block = 4 columns, rows = j1), 64 instructions;
//   * C goes through a per-wave LDS tile (padded) into the A operand of
//     stage 2, C' = (j1 j2) x b = 16 x 32;
//   * stage 2, E_u = C'.D_u for two rows at a time with v_mfma_f32_16x16x4f32
//     (N = 2 rows x 8 columns), 8 instructions per pair.
// ---------------------------------------------------------------------------
constexpr int F32_WAVES = 4;
constexpr int F32_CSTRIDE = 33;              // padded b stride of the C tile
constexpr int F32_CTILE = 4 * 4 * F32_CSTRIDE;  // floats per wave

__device__ __forceinline__ void f32_load_A(const float* G1, int t, int i1, int n1, int lane, float* A) {
  const float4* Ag = reinterpret_cast<const float4*>(G1 + (int64_t)(t * n1 + i1) * 128 + (lane & 3) * 32);
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    float4 v = Ag[m];
    A[4 * m + 0] = v.x;
    A[4 * m + 1] = v.y;
    A[4 * m + 2] = v.z;
    A[4 * m + 3] = v.w;
  }
}

__global__ void __launch_bounds__(64 * F32_WAVES, 3) k_fwd_r32(ShapeArgs s, const float* __restrict__ G1,
                                                           const float* __restrict__ G2,
                                                           const float* __restrict__ G3,
                                                           const int4* __restrict__ slices,
                                                           const uint32_t* __restrict__ uniq_key,
                                                           int32_t* __restrict__ ctr, float* __restrict__ E) {
  __shared__ float ctile[F32_WAVES][F32_CTILE];
  const int lane = lane_id();
  const int wv = threadIdx.x >> 6;
  float* Ct = ctile[wv];
  const int me = blockIdx.x * F32_WAVES + wv;
  const int nworkers = gridDim.x * F32_WAVES;
  const int nsl = ctr[C_NSLICES];
  const int nchunks = (nsl + FWD_CHUNK - 1) / FWD_CHUNK;
  int victim = 0;
  int cur_ti2 = -1, cur_pg = -1;
  float Bl[32], Bh[32];  // B[k][lane], B[k][lane + 64]
  float Cop[8];          // stage-2 A operand: C'[lane % 16][4 s + lane / 16]
  const int jr = (lane & 15) >> 2, j2r = lane & 3, kq = lane >> 4;  // C' read coordinates
  const int sel = (lane & 15) >> 3, j3 = lane & 7;                    // stage-2 B operand / output column
  while (true) {
    const int c = claim_chunk_wave(ctr + C_FWD_CTR, ctr + C_FWD_STEAL, nchunks, nworkers, me, &victim);
    if (c < 0) break;
    const int s0 = c * FWD_CHUNK;
    const int ns = (s0 + FWD_CHUNK < nsl ? s0 + FWD_CHUNK : nsl) - s0;
    // the chunk's slice descriptors, one per lane
    int4 myd = make_int4(0, 0, 0, 0);
    if (lane < ns) myd = slices[s0 + lane];
    // prefetch of slice 0: A and the uniq keys of its rows (lane r holds row rb + r)
    float An[32];
    uint32_t keyn = 0;
    {
      const int p = __shfl(myd.x, 0, 64), rb = __shfl(myd.y, 0, 64), re = __shfl(myd.z, 0, 64);
      const uint32_t key = (uint32_t)__shfl(myd.w, 0, 64);
      const int t = key / s.n12, q = key % s.n12;
      if (p != cur_pg) f32_load_A(G1, t, q / s.n2, s.n1, lane, An);
      if (lane < re - rb) keyn = uniq_key[rb + lane];
    }
    for (int j = 0; j < ns; ++j) {
      const int p = __shfl(myd.x, j, 64), rb = __shfl(myd.y, j, 64), re = __shfl(myd.z, j, 64);
      const uint32_t key = (uint32_t)__shfl(myd.w, j, 64);
      const int t = key / s.n12, q = key % s.n12;
      const int i2 = q % s.n2;
      const int ti2 = t * s.n2 + i2;
      const int i3c = decode_key(keyn, s.Npad, s.n2, s.n3).i3;  // i3 of row rb + lane
      const bool need_c = p != cur_pg;
      if (ti2 != cur_ti2) {
        const float* Bg = G2 + (int64_t)ti2 * 4096;
#pragma unroll
        for (int k = 0; k < 32; ++k) {
          Bl[k] = Bg[k * 128 + lane];
          Bh[k] = Bg[k * 128 + 64 + lane];
        }
        cur_ti2 = ti2;
      }
      if (need_c) {
        f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 32; ++k) {
          c0 = __builtin_amdgcn_mfma_f32_4x4x1f32(An[k], Bl[k], c0, 0, 0, 0);
          c1 = __builtin_amdgcn_mfma_f32_4x4x1f32(An[k], Bh[k], c1, 0, 0, 0);
        }
        // lane holds C[j1 = r][col = lane + 64 h], col = j2 * 32 + b
        wave_lds_sync();
        const int b = lane & 31, j2lo = lane >> 5;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          Ct[r * (4 * F32_CSTRIDE) + j2lo * F32_CSTRIDE + b] = c0[r];
          Ct[r * (4 * F32_CSTRIDE) + (j2lo + 2) * F32_CSTRIDE + b] = c1[r];
        }
        wave_lds_sync();
#pragma unroll
        for (int q4 = 0; q4 < 8; ++q4) Cop[q4] = Ct[jr * (4 * F32_CSTRIDE) + j2r * F32_CSTRIDE + 4 * q4 + kq];
        cur_pg = p;
      }
      // prefetch slice j + 1 (its A once this one's stage 1 is done, and its row keys)
      if (j + 1 < ns) {
        const int pn = __shfl(myd.x, j + 1, 64), rbn = __shfl(myd.y, j + 1, 64), ren = __shfl(myd.z, j + 1, 64);
        const uint32_t kn = (uint32_t)__shfl(myd.w, j + 1, 64);
        const int tn = kn / s.n12, qn = kn % s.n12;
        if (pn != p) f32_load_A(G1, tn, qn / s.n2, s.n1, lane, An);
        keyn = lane < ren - rbn ? uniq_key[rbn + lane] : 0u;
      }
      // rows in pairs; G3 operands of the next pair are loaded before this pair's MFMAs
      const int nr = re - rb;
      const float* G3t = G3 + (int64_t)t * s.n3 * 256;
      auto load_pair = [&](int r0, float* Dv) {
        const bool has1 = r0 + 1 < nr;
        const int rr = sel ? (has1 ? r0 + 1 : r0) : r0;
        const int i3 = __shfl(i3c, rr, 64);
        const float* Dg = G3t + i3 * 256;
        const bool live = !sel || has1;
#pragma unroll
        for (int q4 = 0; q4 < 8; ++q4) Dv[q4] = live ? Dg[(4 * q4 + kq) * 8 + j3] : 0.f;
      };
      float Dc[8], Dn[8];
      load_pair(0, Dc);
      for (int r0 = 0; r0 < nr; r0 += 2) {
        if (r0 + 2 < nr) load_pair(r0 + 2, Dn);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q4 = 0; q4 < 8; ++q4) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(Cop[q4], Dc[q4], acc, 0, 0, 0);
        const bool has1 = r0 + 1 < nr;
        if (!sel || has1) {
          float* Eo = E + (int64_t)(rb + r0 + sel) * 128 + (4 * kq) * 8 + j3;
#pragma unroll
          for (int r = 0; r < 4; ++r) Eo[r * 8] = acc[r];
        }
#pragma unroll
        for (int q4 = 0; q4 < 8; ++q4) Dc[q4] = Dn[q4];
      }
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
  if (s.D % 4 == 0) {
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

hipError_t launch_forward(const Shape& s, const Work& w, const float* G1, const float* G2, const float* G3,
                          const int64_t* offsets, int64_t M, int64_t B, float* out, const Prof& prof,
                          hipStream_t st) {
  if (M > 0) {
    const int grid = persistent_grid() * 2;
    hipError_t e = fill_u32(reinterpret_cast<uint32_t*>(w.ctr + C_FWD_CTR), MAX_PERSIST_WG, 0u, st);
    if (e != hipSuccess) return e;
    e = fill_u32(reinterpret_cast<uint32_t*>(w.ctr + C_FWD_STEAL), 1, 0u, st);
    if (e != hipSuccess) return e;
    if (s.d1 == 4 && s.d2 == 4 && s.d3 == 8 && s.R == 32) {
      const int blocks = (persistent_grid() * 12) / F32_WAVES;
      prof_begin(prof, K_FWD_FUSED, st);
      hipLaunchKernelGGL(k_fwd_r32, dim3(blocks), dim3(64 * F32_WAVES), 0, st, shape_args(s), G1, G2, G3,
                         (const int4*)w.slices, (const uint32_t*)w.uniq_key, w.ctr, w.E);
      prof_end(prof, K_FWD_FUSED, st);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      return launch_pool(s, w.E, w.inv, offsets, M, B, out, prof, st);
    }
    const size_t lds = sizeof(float) * (size_t)s.d1 * s.d2 * s.R;
    e = hipFuncSetAttribute((const void*)k_fwd_generic, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    prof_begin(prof, K_FWD_FUSED, st);
    hipLaunchKernelGGL(k_fwd_generic, dim3(grid), dim3(FWD_THREADS), lds, st, shape_args(s), G1, G2, G3,
                       (const int4*)w.slices, (const uint32_t*)w.uniq_key, w.ctr, w.E);
    prof_end(prof, K_FWD_FUSED, st);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return launch_pool(s, w.E, w.inv, offsets, M, B, out, prof, st);
}

}  // namespace ttemb
