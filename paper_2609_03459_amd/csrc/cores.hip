// TT embeddings with L != 3 cores (Eq. 2 takes any number of row factors; the
// paper leaves L > 3 to future work).  The row is rebuilt by the chain of the L
// core slices, X_0 = S_0 and X_k = X_{k-1} . S_k, and the prefix of Section 3.3
// becomes the first L-1 digits.
//
// The grouping and the fused kernels work on a three-factor view of the shape.
// For L >= 4 the first L-2 cores are contracted into a merged first core
//     G1m[t][i1'] = S_0 . S_1 . ... . S_{L-3}   (d1' x R, d1' = d_0 ... d_{L-3})
// for every i1' = (i_0, ..., i_{L-3}) of every table.  Cores L-2 and L-1 are
// the view's second and third cores, so per prefix group the fused forward
// builds C = G1m[i1'] . S_{L-2} once and E = C . S_{L-1} per row, as for three
// cores: the prefix is the first L-1 digits, and the product of the first L-2
// digits is built once per distinct value rather than once per group.  The
// backward of the view yields dG1m, which goes back through the chain (Eq. 1
// applied to each product in turn) into the gradients of cores 0..L-3.  For
// L = 2 the view's middle core is the identity.
#include "common.h"

namespace ttemb {

constexpr int LV_THREADS = 256;

// Per table, level k (k = 0..K-1, K = L-2 merged cores) holds the partial
// product X_k(q) = S_0[i_0] . ... . S_k[i_k] of every prefix q = (i_0, ..., i_k)
// of the merged digits: P_{k+1} = n_0 ... n_k rows of m_k x R floats,
// m_k = d_0 ... d_k.  Level 0 is core 0 itself and level K-1 is the merged core.
// Each level is built once from its parent level (prefix reuse down the chain),
// and the gradient goes back one level at a time:
//   dS_k[c]      = sum over parents p of X_{k-1}(p)^T . dX_k(p n_k + c)
//   dX_{k-1}(p)  = sum over children c of dX_k(p n_k + c) . S_k[c]^T
// with dX_{K-1} the merged core's gradient and dS_0 = dX_0.
struct LevelArgs {
  int T, R;
  int nk;         // children per parent: n_k
  int64_t P;      // parents per table: P_k = n_0 ... n_{k-1}
  int mprev;      // rows of a parent product: m_{k-1}
  int cols;       // d_k R
};

static LevelArgs level_args(const Shape& s, int k) {
  LevelArgs a;
  a.T = s.T;
  a.R = s.R;
  a.nk = s.nk[k];
  a.P = 1;
  a.mprev = 1;
  for (int j = 0; j < k; ++j) {
    a.P *= s.nk[j];
    a.mprev *= s.dk[j];
  }
  a.cols = s.dk[k] * s.R;
  return a;
}

int64_t core_elems(const Shape& s, int k) {
  const int64_t rl = k == 0 ? 1 : s.R, rr = k == s.L - 1 ? 1 : s.R;
  return (int64_t)s.T * s.nk[k] * rl * s.dk[k] * rr;
}

// Floats of the inner levels 1..K-2 (one region for the products, one for
// their gradients); level k starts at level_offset(s, k).
static int64_t level_offset(const Shape& s, int k) {
  int64_t off = 0, P = s.nk[0], m = s.dk[0];
  for (int j = 1; j < k; ++j) {
    P *= s.nk[j];
    m *= s.dk[j];
    off += (int64_t)s.T * P * m * s.R;
  }
  return off;
}

int64_t chain_level_floats(const Shape& s) { return s.L >= 5 ? level_offset(s, s.L - 3) : 0; }

// X_k(t, p n_k + c) = X_{k-1}(t, p) . S_k(t, c).  Block (t, c, chunk) takes
// child c and a chunk of pc consecutive parents: their rows X_{k-1} and the
// slice S_k(t, c) (padded rows) are staged in LDS, and each thread forms
// output columns of the chunk's products.
__global__ void __launch_bounds__(LV_THREADS) k_merge_level(LevelArgs a, int pc, int stage_s,
                                                            const float* __restrict__ Xprev,
                                                            const float* __restrict__ Sk, float* __restrict__ Xk) {
  extern __shared__ float lds[];
  const int64_t nchunk = (a.P + pc - 1) / pc;
  const int64_t tc = blockIdx.x / nchunk;  // t * n_k + c
  const int64_t p0 = (blockIdx.x - tc * nchunk) * pc;
  const int64_t t = tc / a.nk;
  const int ch = (int)(tc - t * a.nk);
  const int np = (int)(a.P - p0 < pc ? a.P - p0 : pc);
  const int xl = a.mprev * a.R, ol = a.mprev * a.cols;
  const int spitch = a.cols + 1;
  float* Xs = lds;
  float* Ss = lds + pc * xl;
  const float* Xg = Xprev + (t * a.P + p0) * xl;
  for (int e = threadIdx.x; e < np * xl; e += LV_THREADS) Xs[e] = Xg[e];
  const float* S = Sk + tc * a.R * a.cols;
  if (stage_s)
    for (int e = threadIdx.x; e < a.R * a.cols; e += LV_THREADS) {
      const int b = e / a.cols, col = e - b * a.cols;
      Ss[b * spitch + col] = S[e];
    }
  __syncthreads();
  const float* Sb = stage_s ? Ss : S;
  const int sp = stage_s ? spitch : a.cols;
  for (int o = threadIdx.x; o < np * ol; o += LV_THREADS) {
    const int pr = o / a.cols, col = o - pr * a.cols;  // pr = pp * mprev + r
    const int pp = pr / a.mprev, r = pr - pp * a.mprev;
    const float* x = Xs + pr * a.R;
    float acc = 0.f;
    for (int b = 0; b < a.R; ++b) acc = fmaf(x[b], Sb[b * sp + col], acc);
    Xk[((t * a.P + p0 + pp) * a.nk + ch) * ol + r * a.cols + col] = acc;
  }
}

// One backward level k of the merged chain.  Block (t, c, chunk) takes child c of
// core k and a chunk of pc consecutive parents p; with X = X_{k-1}(t, p) and
// dX = dX_k(t, p n_k + c) staged in LDS it writes
//     X^T . dX              summed over the chunk: the (t, c, chunk) partial of dS_k(t, c)
//     dX . S_k(t, c)^T      for each parent: the (t, p, c) partial of dX_{k-1}(t, p)
// No two blocks write one partial; k_split_sum adds them in a fixed order.
__global__ void __launch_bounds__(LV_THREADS) k_split_level(LevelArgs a, int pc, int stage_s,
                                                            const float* __restrict__ Xprev,
                                                            const float* __restrict__ dXk,
                                                            const float* __restrict__ Sk, float* __restrict__ partS,
                                                            float* __restrict__ partX) {
  extern __shared__ float lds[];
  const int64_t nchunk = (a.P + pc - 1) / pc;
  const int64_t tc = blockIdx.x / nchunk;  // t * n_k + c
  const int64_t p0 = (blockIdx.x - tc * nchunk) * pc;
  const int64_t t = tc / a.nk;
  const int ch = (int)(tc - t * a.nk);
  const int np = (int)(a.P - p0 < pc ? a.P - p0 : pc);
  const int xl = a.mprev * a.R, dl = a.mprev * a.cols;
  const int spitch = a.cols + 1;
  float* Xs = lds;
  float* dXs = Xs + pc * xl;
  float* Ss = dXs + pc * dl;
  const float* S = Sk + tc * a.R * a.cols;
  const float* Xg = Xprev + (t * a.P + p0) * xl;  // consecutive parents are contiguous
  for (int e = threadIdx.x; e < np * xl; e += LV_THREADS) Xs[e] = Xg[e];
  for (int e = threadIdx.x; e < np * dl; e += LV_THREADS) {
    const int pp = e / dl, w = e - pp * dl;
    dXs[e] = dXk[((t * a.P + p0 + pp) * a.nk + ch) * dl + w];
  }
  if (stage_s)
    for (int e = threadIdx.x; e < a.R * a.cols; e += LV_THREADS) {
      const int b = e / a.cols, col = e - b * a.cols;
      Ss[b * spitch + col] = S[e];
    }
  __syncthreads();
  const int rows = np * a.mprev;
  float* gS = partS + blockIdx.x * (int64_t)a.R * a.cols;  // blockIdx.x = tc * nchunk + chunk
  for (int o = threadIdx.x; o < a.R * a.cols; o += LV_THREADS) {
    const int b = o / a.cols, col = o - b * a.cols;
    float acc = 0.f;
    for (int r = 0; r < rows; ++r) acc = fmaf(Xs[r * a.R + b], dXs[r * a.cols + col], acc);
    gS[o] = acc;
  }
  for (int o = threadIdx.x; o < rows * a.R; o += LV_THREADS) {
    const int r = o / a.R, b = o - r * a.R;
    const int pp = r / a.mprev, rr = r - pp * a.mprev;
    const float* d = dXs + r * a.cols;
    float acc = 0.f;
    if (stage_s) {
      const float* sr = Ss + b * spitch;
      for (int col = 0; col < a.cols; ++col) acc = fmaf(d[col], sr[col], acc);
    } else {
      const float* sr = S + b * a.cols;
      for (int col = 0; col < a.cols; ++col) acc = fmaf(d[col], sr[col], acc);
    }
    partX[((t * a.P + p0 + pp) * a.nk + ch) * xl + rr * a.R + b] = acc;
  }
}

// dS_k(t, c) = sum over the parent chunks of their partials (chunk order), and
// dX_{k-1}(t, p) = sum over the children c of their partials (c ascending): one
// thread per output element, elements [0, nS) of dS_k then [0, nX) of dX_{k-1}.
__global__ void __launch_bounds__(LV_THREADS) k_split_sum(LevelArgs a, int64_t nchunk,
                                                          const float* __restrict__ partS,
                                                          const float* __restrict__ partX, float* __restrict__ dSk,
                                                          float* __restrict__ dXprev) {
  const int64_t RC = (int64_t)a.R * a.cols, xl = (int64_t)a.mprev * a.R;
  const int64_t nS = (int64_t)a.T * a.nk * RC, nX = (int64_t)a.T * a.P * xl;
  for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < nS + nX; o += (int64_t)gridDim.x * blockDim.x) {
    float acc = 0.f;
    if (o < nS) {
      const int64_t tc = o / RC, e = o - tc * RC;
      for (int64_t j = 0; j < nchunk; ++j) acc += partS[(tc * nchunk + j) * RC + e];
      dSk[o] = acc;
    } else {
      const int64_t x = o - nS;
      const int64_t tp = x / xl, w = x - tp * xl;
      for (int c = 0; c < a.nk; ++c) acc += partX[(tp * a.nk + c) * xl + w];
      dXprev[x] = acc;
    }
  }
}

// Parents per block of the split of level k: their X and dX rows within 32 KB of
// LDS, and whether S_k(t, c) (padded rows) is staged too (16 KB more).
static void split_plan(const Shape& s, int k, int64_t* pc_out, int* stage_out) {
  const LevelArgs a = level_args(s, k);
  const int64_t per = (int64_t)a.mprev * (a.R + a.cols);
  int64_t pc = 8192 / per;
  if (pc < 1) pc = 1;
  if (pc > a.P) pc = a.P;
  *pc_out = pc;
  *stage_out = (int64_t)a.R * (a.cols + 1) <= 4096;
}

int64_t split_partial_floats(const Shape& s) {
  int64_t most = 0;
  for (int k = 1; k <= s.L - 3; ++k) {
    const LevelArgs a = level_args(s, k);
    int64_t pc;
    int st;
    split_plan(s, k, &pc, &st);
    const int64_t nchunk = (a.P + pc - 1) / pc;
    const int64_t n = (int64_t)a.T * a.nk * nchunk * a.R * a.cols + (int64_t)a.T * a.P * a.nk * a.mprev * a.R;
    if (n > most) most = n;
  }
  return most;
}

__global__ void k_identity(float* __restrict__ G, int T, int R) {
  const int64_t n = (int64_t)T * R * R;
  for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < n; o += (int64_t)gridDim.x * blockDim.x) {
    const int64_t e = o % ((int64_t)R * R);
    G[o] = (e / R == e % R) ? 1.f : 0.f;
  }
}

// Product level k (1..K-1): the merged core for k = K-1, else an inner level.
static float* level_x(const Shape& s, const Work& w, int k) {
  return k == s.L - 3 ? w.g1m : w.xlev + level_offset(s, k);
}

hipError_t launch_merge(const Shape& s, const Work& w, const float* const* cores, const Prof& prof, hipStream_t st) {
  if (s.L < 4 || !w.g1m || (s.L >= 5 && !w.xlev)) return hipErrorInvalidValue;
  prof_begin(prof, K_MERGE, st);
  for (int k = 1; k <= s.L - 3; ++k) {
    const LevelArgs a = level_args(s, k);
    const float* Xprev = k == 1 ? cores[0] : level_x(s, w, k - 1);
    // S_k(t, c) staged (padded rows) when it fits in 32 KB; parents per block:
    // 16, fewer if their rows and the staged slice exceed 48 KB of LDS
    const int stage_s = (int64_t)a.R * (a.cols + 1) <= 8192;
    const int64_t sl = stage_s ? (int64_t)a.R * (a.cols + 1) : 0, xl = (int64_t)a.mprev * a.R;
    int64_t pc = (12288 - sl) / xl;
    if (pc > 16) pc = 16;
    if (pc < 1) pc = 1;
    if (pc > a.P) pc = a.P;
    const size_t lds = sizeof(float) * (size_t)(pc * xl + sl);
    hipError_t e = hipFuncSetAttribute((const void*)k_merge_level, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
    const int64_t blocks = (int64_t)a.T * a.nk * ((a.P + pc - 1) / pc);
    hipLaunchKernelGGL(k_merge_level, dim3((unsigned)blocks), dim3(LV_THREADS), lds, st, a, (int)pc, stage_s,
                       Xprev, cores[k], level_x(s, w, k));
  }
  prof_end(prof, K_MERGE, st);
  return hipGetLastError();
}

hipError_t launch_split(const Shape& s, const Work& w, const float* const* cores, float* const* grads,
                        const Prof& prof, hipStream_t st) {
  if (s.L < 4 || !w.g1m || !w.dg1m || !w.splitpart || (s.L >= 5 && (!w.xlev || !w.dxlev)))
    return hipErrorInvalidValue;
  hipError_t e;
  prof_begin(prof, K_SPLIT, st);
  for (int k = s.L - 3; k >= 1; --k) {
    const LevelArgs a = level_args(s, k);
    const float* Xprev = k == 1 ? cores[0] : level_x(s, w, k - 1);
    const float* dXk = k == s.L - 3 ? w.dg1m : w.dxlev + level_offset(s, k);
    float* dXprev = k == 1 ? grads[0] : w.dxlev + level_offset(s, k - 1);
    int64_t pc;
    int stage_s;
    split_plan(s, k, &pc, &stage_s);
    const int64_t per = (int64_t)a.mprev * (a.R + a.cols);
    const size_t lds = sizeof(float) * (size_t)(pc * per + (stage_s ? a.R * (a.cols + 1) : 0));
    if ((e = hipFuncSetAttribute((const void*)k_split_level, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)lds)) != hipSuccess)
      return e;
    const int64_t nchunk = (a.P + pc - 1) / pc;
    const int64_t blocks = (int64_t)a.T * a.nk * nchunk;
    float* partS = w.splitpart;
    float* partX = partS + blocks * a.R * a.cols;
    hipLaunchKernelGGL(k_split_level, dim3((unsigned)blocks), dim3(LV_THREADS), lds, st, a, (int)pc, stage_s, Xprev,
                       dXk, (const float*)cores[k], partS, partX);
    const int64_t nout = (int64_t)a.T * a.nk * a.R * a.cols + (int64_t)a.T * a.P * a.mprev * a.R;
    int64_t sb = (nout + LV_THREADS - 1) / LV_THREADS;
    if (sb > 8192) sb = 8192;
    hipLaunchKernelGGL(k_split_sum, dim3((unsigned)sb), dim3(LV_THREADS), 0, st, a, nchunk, (const float*)partS,
                       (const float*)partX, grads[k], dXprev);
  }
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
