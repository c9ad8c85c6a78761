// TT embeddings with L != 3 cores (Eq. 2 takes any number of row factors; the
// paper leaves L > 3 to future work).  The row is rebuilt by the chain of the L
// core slices, X_0 = S_0 and X_k = X_{k-1} . S_k, and the prefix of Section 3.3
// becomes the first L-1 digits.
//
// The grouping and the fused kernels work on a three-factor view of the shape.
// For L >= 4 the first L-2 cores are contracted into a merged first core
//     G1m[t][i1'] = S_0 . S_1 . ... . S_{L-3}   (d1' x R, d1' = d_0 ... d_{L-3})
// for every i1' = (i_0, ..., i_{L-3}) of every table (k_merge).  Cores L-2 and
// L-1 are the view's second and third cores, so per prefix group the fused
// forward builds C = G1m[i1'] . S_{L-2} once and E = C . S_{L-1} per row, as
// for three cores: the prefix is the first L-1 digits, and the product of the
// first L-2 digits is built once per distinct value rather than once per group.
// The backward of the view yields dG1m; k_split carries it back through the
// chain (Eq. 1 applied to each product in turn) into the gradients of cores
// 0..L-3.  For L = 2 the view's middle core is the identity.
#include "common.h"

namespace ttemb {

constexpr int CH_THREADS = 128;

struct ChainArgs {
  int T, K, R;        // K = L - 2 merged cores
  int n1v, d1v;       // their row and column products
  int n[MAX_CORES];   // row factors of the merged cores
  int d[MAX_CORES];   // column factors
  int rstride[MAX_CORES];  // digit k of i1' is (i1' / rstride[k]) mod n[k]
};

struct CorePtrs {
  const float* p[MAX_CORES];
};
struct GradPtrs {
  float* p[MAX_CORES];
};

static ChainArgs chain_args(const Shape& s) {
  ChainArgs a;
  a.T = s.T;
  a.K = s.L - 2;
  a.R = s.R;
  a.n1v = s.n1;
  a.d1v = s.d1;
  int stride = 1;
  for (int k = MAX_CORES - 1; k >= 0; --k) {
    const bool in = k < a.K;
    a.n[k] = in ? s.nk[k] : 1;
    a.d[k] = in ? s.dk[k] : 1;
    a.rstride[k] = in ? stride : 1;
    if (in) stride *= s.nk[k];
  }
  return a;
}

int64_t core_elems(const Shape& s, int k) {
  const int64_t rl = k == 0 ? 1 : s.R, rr = k == s.L - 1 ? 1 : s.R;
  return (int64_t)s.T * s.nk[k] * rl * s.dk[k] * rr;
}

// LDS of the split kernel (the larger of the two): X_0 .. X_{K-2} plus two dX
// buffers of d1' x R; the merge kernel needs two buffers of d1' x R.
int64_t chain_lds_floats(const Shape& s) {
  if (s.L < 4) return 0;
  int64_t m = 1, xs = 0;
  for (int k = 0; k + 1 < s.L - 2; ++k) {
    m *= s.dk[k];
    xs += m * s.R;
  }
  return xs + 2 * (int64_t)s.d1 * s.R;
}

// Slice S_k of table t at digit i: r_k x (d_k r_{k+1}) floats; r_0 = 1, else R.
__device__ __forceinline__ const float* chain_slice(const ChainArgs& a, const float* G, int k, int t, int i) {
  const int64_t len = (int64_t)(k == 0 ? 1 : a.R) * a.d[k] * a.R;
  return G + ((int64_t)t * a.n[k] + i) * len;
}

// out (m x cols) = X (m x R) . S (R x cols), X in LDS, S in global memory.
__device__ __forceinline__ void chain_mul(const float* X, const float* __restrict__ S, float* out, int m, int R,
                                          int cols) {
  for (int o = threadIdx.x; o < m * cols; o += CH_THREADS) {
    const int r = o / cols, c = o - r * cols;
    float acc = 0.f;
    for (int b = 0; b < R; ++b) acc = fmaf(X[r * R + b], S[b * cols + c], acc);
    out[o] = acc;
  }
}

// One block per (table, i1'): G1m[t][i1'] = S_0 . ... . S_{K-1}.
__global__ void __launch_bounds__(CH_THREADS) k_merge(ChainArgs a, CorePtrs G, float* __restrict__ G1m) {
  extern __shared__ float lds[];
  const int row = blockIdx.x;
  const int t = row / a.n1v, i1 = row - t * a.n1v;
  float* X = lds;
  float* Y = lds + a.d1v * a.R;
  const float* S0 = chain_slice(a, G.p[0], 0, t, (i1 / a.rstride[0]) % a.n[0]);
  int m = a.d[0];
  for (int o = threadIdx.x; o < m * a.R; o += CH_THREADS) X[o] = S0[o];
  for (int k = 1; k < a.K; ++k) {
    __syncthreads();
    const float* S = chain_slice(a, G.p[k], k, t, (i1 / a.rstride[k]) % a.n[k]);
    float* out = k == a.K - 1 ? G1m + (int64_t)row * a.d1v * a.R : Y;
    chain_mul(X, S, out, m, a.R, a.d[k] * a.R);
    float* tmp = X;
    X = Y;
    Y = tmp;
    m *= a.d[k];
  }
}

// One block per (table, i1'): the gradient dX_{K-1} = dG1m[t][i1'] goes back
// through the chain; per product X_k = X_{k-1} . S_k,
//     dS_k += X_{k-1}^T . dX_k   and   dX_{k-1} = dX_k . S_k^T
// (dX_k viewed as m_{k-1} x (d_k R)), and finally dS_0 += dX_0.  Core
// gradients of slices shared by several i1' meet in global atomics.  A row with
// an all-zero gradient (no index reached it) adds nothing and is skipped.
__global__ void __launch_bounds__(CH_THREADS) k_split(ChainArgs a, CorePtrs G, GradPtrs dG,
                                                      const float* __restrict__ dG1m) {
  extern __shared__ float lds[];
  const int row = blockIdx.x;
  const int t = row / a.n1v, i1 = row - t * a.n1v;
  const int nd = a.d1v * a.R;
  float* dX = lds;
  float* dY = lds + nd;
  float* Xs = lds + 2 * nd;  // X_0, X_1, ... X_{K-2}, packed
  const float* g = dG1m + (int64_t)row * nd;
  int nz = 0;
  for (int o = threadIdx.x; o < nd; o += CH_THREADS) {
    const float v = g[o];
    dX[o] = v;
    nz |= v != 0.f;
  }
  if (!__syncthreads_or(nz)) return;
  // X_0 .. X_{K-2}
  const float* S0 = chain_slice(a, G.p[0], 0, t, (i1 / a.rstride[0]) % a.n[0]);
  int m = a.d[0];
  for (int o = threadIdx.x; o < m * a.R; o += CH_THREADS) Xs[o] = S0[o];
  float* Xk = Xs;
  for (int k = 1; k + 1 < a.K; ++k) {
    __syncthreads();
    const float* S = chain_slice(a, G.p[k], k, t, (i1 / a.rstride[k]) % a.n[k]);
    chain_mul(Xk, S, Xk + m * a.R, m, a.R, a.d[k] * a.R);
    Xk += m * a.R;
    m *= a.d[k];
  }
  // Xk = X_{K-2} (m = m_{K-2} rows)
  for (int k = a.K - 1; k >= 1; --k) {
    __syncthreads();
    const int cols = a.d[k] * a.R;
    const int ik = (i1 / a.rstride[k]) % a.n[k];
    const float* S = chain_slice(a, G.p[k], k, t, ik);
    float* gk = dG.p[k] + ((int64_t)t * a.n[k] + ik) * a.R * cols;
    for (int o = threadIdx.x; o < a.R * cols; o += CH_THREADS) {
      const int b = o / cols, c = o - b * cols;
      float acc = 0.f;
      for (int r = 0; r < m; ++r) acc = fmaf(Xk[r * a.R + b], dX[r * cols + c], acc);
      unsafeAtomicAdd(&gk[o], acc);
    }
    for (int o = threadIdx.x; o < m * a.R; o += CH_THREADS) {
      const int r = o / a.R, b = o - r * a.R;
      float acc = 0.f;
      for (int c = 0; c < cols; ++c) acc = fmaf(dX[r * cols + c], S[b * cols + c], acc);
      dY[o] = acc;
    }
    float* tmp = dX;
    dX = dY;
    dY = tmp;
    if (k > 1) {
      m /= a.d[k - 1];
      Xk -= m * a.R;
    }
  }
  __syncthreads();
  const int i0 = (i1 / a.rstride[0]) % a.n[0];
  float* g0 = dG.p[0] + ((int64_t)t * a.n[0] + i0) * a.d[0] * a.R;
  for (int o = threadIdx.x; o < a.d[0] * a.R; o += CH_THREADS) unsafeAtomicAdd(&g0[o], dX[o]);
}

__global__ void k_identity(float* __restrict__ G, int T, int R) {
  const int64_t n = (int64_t)T * R * R;
  for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < n; o += (int64_t)gridDim.x * blockDim.x) {
    const int64_t e = o % ((int64_t)R * R);
    G[o] = (e / R == e % R) ? 1.f : 0.f;
  }
}

static CorePtrs core_ptrs(const float* const* cores, int K) {
  CorePtrs c;
  for (int k = 0; k < MAX_CORES; ++k) c.p[k] = k < K ? cores[k] : nullptr;
  return c;
}

hipError_t launch_merge(const Shape& s, const Work& w, const float* const* cores, const Prof& prof, hipStream_t st) {
  if (s.L < 4 || !w.g1m) return hipErrorInvalidValue;
  const ChainArgs a = chain_args(s);
  const size_t lds = sizeof(float) * 2 * (size_t)s.d1 * s.R;
  hipError_t e = hipFuncSetAttribute((const void*)k_merge, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  prof_begin(prof, K_MERGE, st);
  hipLaunchKernelGGL(k_merge, dim3((unsigned)((int64_t)s.T * s.n1)), dim3(CH_THREADS), lds, st, a,
                     core_ptrs(cores, a.K), w.g1m);
  prof_end(prof, K_MERGE, st);
  return hipGetLastError();
}

hipError_t launch_split(const Shape& s, const Work& w, const float* const* cores, float* const* grads,
                        const Prof& prof, hipStream_t st) {
  if (s.L < 4 || !w.dg1m) return hipErrorInvalidValue;
  const ChainArgs a = chain_args(s);
  hipError_t e;
  for (int k = 0; k < a.K; ++k)
    if ((e = fill_f32(grads[k], core_elems(s, k), 0.f, st)) != hipSuccess) return e;
  const size_t lds = sizeof(float) * (size_t)chain_lds_floats(s);
  if ((e = hipFuncSetAttribute((const void*)k_split, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) !=
      hipSuccess)
    return e;
  GradPtrs g;
  for (int k = 0; k < MAX_CORES; ++k) g.p[k] = k < a.K ? grads[k] : nullptr;
  prof_begin(prof, K_SPLIT, st);
  hipLaunchKernelGGL(k_split, dim3((unsigned)((int64_t)s.T * s.n1)), dim3(CH_THREADS), lds, st, a,
                     core_ptrs(cores, a.K), g, (const float*)w.dg1m);
  prof_end(prof, K_SPLIT, st);
  return hipGetLastError();
}

hipError_t launch_identity(const Shape& s, const Work& w, hipStream_t st) {
  if (s.L != 2 || !w.g1m) return hipErrorInvalidValue;
  const int64_t n = (int64_t)s.T * s.R * s.R;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(k_identity, dim3((unsigned)blocks), dim3(256), 0, st, w.g1m, s.T, s.R);
  return hipGetLastError();
}

}  // namespace ttemb
