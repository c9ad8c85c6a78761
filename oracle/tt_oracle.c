/*
 * Plain CPU oracle for the Tensor-Train (TT) embedding gather.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the correctness reference that the
 * GPU library is checked against.  Only the test suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it; the product path never
 * does.  It shares no code, header, table or helper with the GPU library.
 *
 * Everything here is the plain definition of the operator, written for a
 * reader holding the paper (FlowTT, ICCAD'26): no deduplication, no prefix
 * reuse, no scheduling.  Each occurrence of a row index is expanded on its
 * own, in position order, and every sum is accumulated in double precision
 * from the float32 inputs.
 *
 * Layouts (float32, row-major, tables contiguous):
 *   G1 [T][n1][d1][R]     slice A = G1[t][i1] is d1 x R
 *   G2 [T][n2][R][d2][R]  slice B = G2[t][i2] is R x (d2 R)
 *   G3 [T][n3][R][d3]     slice D = G3[t][i3] is R x d3
 *   pooled output V [T][B][D] with D = d1 d2 d3 and the output digit j1 most
 *   significant: E[j1*d2*d3 + j2*d3 + j3].
 * Bags: offsets is a CSR array of T*B+1 entries over the concatenated index
 * array; bag gb = t*B + b of table t covers idx[offsets[gb] .. offsets[gb+1]).
 * A NULL offsets array means one index per bag (idx has T*B entries).
 * An index outside [0, N) contributes nothing and is counted as invalid.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Mixed-radix conversion, Eq. 2 (Section 3.3): the k-th digit of g is
 * floor(g / prod_{j>k} p_j) mod p_k, the first factor being the most
 * significant digit. */
static void mixed_radix3(int64_t g, const int32_t n[3], int64_t dig[3]) {
  for (int k = 0; k < 3; ++k) {
    int64_t prod = 1;
    for (int j = k + 1; j < 3; ++j) prod *= n[j];
    dig[k] = (g / prod) % n[k];
  }
}

void orc_digits(const int64_t* g, int64_t m, const int32_t n[3], int64_t* out /* [m][3] */) {
  for (int64_t o = 0; o < m; ++o) mixed_radix3(g[o], n, out + 3 * o);
}

typedef struct {
  int T;
  int64_t N;
  int32_t n[3];
  int32_t d[3];
  int R;
  int64_t B;
} shape_t;

static int64_t dimD(const shape_t* s) { return (int64_t)s->d[0] * s->d[1] * s->d[2]; }

/* Table and bag of every occurrence, from the CSR offsets (or the identity). */
static void bag_of_occurrences(const shape_t* s, int64_t M, const int64_t* offsets, int64_t* bag) {
  int64_t nb = (int64_t)s->T * s->B;
  if (!offsets) {
    for (int64_t o = 0; o < M; ++o) bag[o] = o;
    return;
  }
  for (int64_t gb = 0; gb < nb; ++gb)
    for (int64_t o = offsets[gb]; o < offsets[gb + 1]; ++o) bag[o] = gb;
}

/* Intermediate C = A . B of Section 3.2 (Fig. 3): A = G1[t][i1] (d1 x R),
 * B = G2[t][i2] (R x d2R); C is d1 x d2R, i.e. (d1 d2) x R row-major. */
static void stage_intermediate(const shape_t* s, const float* A, const float* Bm, double* C) {
  int d1 = s->d[0], d2 = s->d[1], R = s->R;
  int cols = d2 * R;
  for (int j1 = 0; j1 < d1; ++j1)
    for (int c = 0; c < cols; ++c) {
      double acc = 0.0;
      for (int a = 0; a < R; ++a) acc += (double)A[j1 * R + a] * (double)Bm[a * cols + c];
      C[j1 * cols + c] = acc;
    }
}

/* Embedding E = C . D of Section 3.2 with C viewed as (d1 d2) x R and
 * D = G3[t][i3] (R x d3). */
static void stage_embedding(const shape_t* s, const double* C, const float* Dm, double* E) {
  int rows = s->d[0] * s->d[1], d3 = s->d[2], R = s->R;
  for (int r = 0; r < rows; ++r)
    for (int j3 = 0; j3 < d3; ++j3) {
      double acc = 0.0;
      for (int b = 0; b < R; ++b) acc += C[r * R + b] * (double)Dm[b * d3 + j3];
      E[r * d3 + j3] = acc;
    }
}

static const float* sliceA(const shape_t* s, const float* G1, int64_t t, int64_t i1) {
  return G1 + ((t * s->n[0] + i1) * s->d[0]) * (int64_t)s->R;
}
static const float* sliceB(const shape_t* s, const float* G2, int64_t t, int64_t i2) {
  return G2 + (t * s->n[1] + i2) * (int64_t)s->R * s->d[1] * s->R;
}
static const float* sliceD(const shape_t* s, const float* G3, int64_t t, int64_t i3) {
  return G3 + (t * s->n[2] + i3) * (int64_t)s->R * s->d[2];
}

/* One embedding row E_g of table t (all D values); C is caller scratch of
 * d1*d2*R doubles. */
static void row_into(const shape_t* s, const float* G1, const float* G2, const float* G3, int64_t t, int64_t g,
                     double* C, double* E) {
  int64_t dig[3];
  mixed_radix3(g, s->n, dig);
  stage_intermediate(s, sliceA(s, G1, t, dig[0]), sliceB(s, G2, t, dig[1]), C);
  stage_embedding(s, C, sliceD(s, G3, t, dig[2]), E);
}

void orc_row(const shape_t* s, const float* G1, const float* G2, const float* G3, int64_t t, int64_t g,
             double* E) {
  double* C = (double*)malloc(sizeof(double) * s->d[0] * s->d[1] * s->R);
  row_into(s, G1, G2, G3, t, g, C, E);
  free(C);
}

/* Forward: V[gb] = sum of E_{idx[o]} over the occurrences o of bag gb
 * (sum pooling; an empty bag gives zero).  If bag_list is non-NULL only the
 * listed global bags are computed and V is [nlist][D] in list order;
 * otherwise V is [T*B][D].  Returns the number of invalid indices met. */
int64_t orc_forward(const shape_t* s, const float* G1, const float* G2, const float* G3, const int64_t* idx,
                    int64_t M, const int64_t* offsets, const int64_t* bag_list, int64_t nlist, double* V) {
  int64_t D = dimD(s);
  int64_t nb = (int64_t)s->T * s->B;
  int64_t count = bag_list ? nlist : nb;
  double* E = (double*)malloc(sizeof(double) * D);
  double* C = (double*)malloc(sizeof(double) * s->d[0] * s->d[1] * s->R);
  int64_t invalid = 0;
  (void)M;
  for (int64_t k = 0; k < count; ++k) {
    int64_t gb = bag_list ? bag_list[k] : k;
    int64_t t = gb / s->B;
    int64_t lo = offsets ? offsets[gb] : gb, hi = offsets ? offsets[gb + 1] : gb + 1;
    double* out = V + k * D;
    for (int64_t j = 0; j < D; ++j) out[j] = 0.0;
    for (int64_t o = lo; o < hi; ++o) {
      int64_t g = idx[o];
      if (g < 0 || g >= s->N) {
        ++invalid;
        continue;
      }
      row_into(s, G1, G2, G3, t, g, C, E);
      for (int64_t j = 0; j < D; ++j) out[j] += E[j];
    }
  }
  free(C);
  free(E);
  return invalid;
}

/* Backward of L = sum_gb <dV[gb], V[gb]> into dense core gradients
 * (overwritten; rows no occurrence touches stay zero).  Every occurrence o,
 * in position order, with dE = dV[bag(o)], adds (Section 3.2, Eq. 1 before
 * regrouping by prefix):
 *   dG3[i3] += C^T dE         (C as (d1 d2) x R, dE as (d1 d2) x d3)
 *   dC       = dE D^T          ((d1 d2) x R, viewed again as d1 x d2R)
 *   dG1[i1] += dC B^T
 *   dG2[i2] += A^T dC
 * Optional masks want1 [T*n1], want2 [T*n2], want3 [T*n3] skip occurrences
 * that touch no wanted slice (the gradients of wanted slices stay exact).
 * Returns the number of invalid indices met. */
int64_t orc_backward(const shape_t* s, const float* G1, const float* G2, const float* G3, const int64_t* idx,
                     int64_t M, const int64_t* offsets, const float* dV, double* dG1, double* dG2, double* dG3,
                     const uint8_t* want1, const uint8_t* want2, const uint8_t* want3) {
  int d1 = s->d[0], d2 = s->d[1], d3 = s->d[2], R = s->R;
  int64_t D = dimD(s);
  int cols = d2 * R;
  int64_t T = s->T;
  memset(dG1, 0, sizeof(double) * T * s->n[0] * d1 * R);
  memset(dG2, 0, sizeof(double) * T * s->n[1] * R * d2 * R);
  memset(dG3, 0, sizeof(double) * T * s->n[2] * R * d3);
  int64_t* bag = (int64_t*)malloc(sizeof(int64_t) * (M > 0 ? M : 1));
  bag_of_occurrences(s, M, offsets, bag);
  double* C = (double*)malloc(sizeof(double) * d1 * cols);
  double* dC = (double*)malloc(sizeof(double) * d1 * cols);
  int64_t invalid = 0;
  for (int64_t o = 0; o < M; ++o) {
    int64_t g = idx[o];
    if (g < 0 || g >= s->N) {
      ++invalid;
      continue;
    }
    int64_t gb = bag[o], t = gb / s->B;
    int64_t dig[3];
    mixed_radix3(g, s->n, dig);
    if (want1 || want2 || want3) {
      int w = (want1 && want1[t * s->n[0] + dig[0]]) || (want2 && want2[t * s->n[1] + dig[1]]) ||
              (want3 && want3[t * s->n[2] + dig[2]]);
      if (!w) continue;
    }
    const float* A = sliceA(s, G1, t, dig[0]);
    const float* Bm = sliceB(s, G2, t, dig[1]);
    const float* Dm = sliceD(s, G3, t, dig[2]);
    const float* dE = dV + gb * D;
    stage_intermediate(s, A, Bm, C);
    /* dG3[i3] += C^T dE */
    double* g3 = dG3 + (t * s->n[2] + dig[2]) * (int64_t)R * d3;
    for (int b = 0; b < R; ++b)
      for (int j3 = 0; j3 < d3; ++j3) {
        double acc = 0.0;
        for (int r = 0; r < d1 * d2; ++r) acc += C[r * R + b] * (double)dE[r * d3 + j3];
        g3[b * d3 + j3] += acc;
      }
    /* dC = dE D^T */
    for (int r = 0; r < d1 * d2; ++r)
      for (int b = 0; b < R; ++b) {
        double acc = 0.0;
        for (int j3 = 0; j3 < d3; ++j3) acc += (double)dE[r * d3 + j3] * (double)Dm[b * d3 + j3];
        dC[r * R + b] = acc;
      }
    /* dG1[i1] += dC B^T, dC as d1 x d2R */
    double* g1 = dG1 + (t * s->n[0] + dig[0]) * (int64_t)d1 * R;
    for (int j1 = 0; j1 < d1; ++j1)
      for (int a = 0; a < R; ++a) {
        double acc = 0.0;
        for (int c = 0; c < cols; ++c) acc += dC[j1 * cols + c] * (double)Bm[a * cols + c];
        g1[j1 * R + a] += acc;
      }
    /* dG2[i2] += A^T dC */
    double* g2 = dG2 + (t * s->n[1] + dig[1]) * (int64_t)R * cols;
    for (int a = 0; a < R; ++a)
      for (int c = 0; c < cols; ++c) {
        double acc = 0.0;
        for (int j1 = 0; j1 < d1; ++j1) acc += (double)A[j1 * R + a] * dC[j1 * cols + c];
        g2[a * cols + c] += acc;
      }
  }
  free(bag);
  free(C);
  free(dC);
  return invalid;
}

/* ---------------------------------------------------------------------------
 * L cores (L >= 2): the same operator with the row split into L mixed-radix
 * digits (Eq. 2 is stated for any number of factors) and the row rebuilt by
 * the chain of the L core slices; the prefix of Section 3.3 becomes the first
 * L-1 digits (deeper decompositions are the paper's stated future work).
 *
 * Core k (k = 0..L-1) is [T][n_k][r_k][d_k][r_{k+1}] with r_0 = r_L = 1 and
 * the other ranks R; its slice S_k = core k [t][i_k] is r_k x (d_k r_{k+1}).
 * The chain: X_0 = S_0 (d_0 x R); X_k = X_{k-1} . S_k with X_{k-1} viewed as
 * m_{k-1} x r_k (m_k = d_0 ... d_k rows), giving m_{k-1} x (d_k r_{k+1}), i.e.
 * m_k x r_{k+1}; X_{L-1} is the row E (D x 1), output digit j_0 most
 * significant.  For L = 3 this is C = A.B (X_1) and E = C.D (X_2).
 * Pinned (CPU tests): equal to the three-core functions above at L = 3; the
 * additive rank-2 train whose row g is g*D + j exactly, for L = 2, 4, 5; an
 * identity middle core that turns L = 4 into L = 3; a float64 torch brute
 * force with autograd gradients; and <dG_k, G_k> = <dV, V> for every k.
 * ------------------------------------------------------------------------- */
#define ORC_MAXL 8

typedef struct {
  int T;
  int64_t N;
  int L;
  int32_t n[ORC_MAXL];
  int32_t d[ORC_MAXL];
  int R;
  int64_t B;
} shape_n_t;

static int rank_n(const shape_n_t* s, int k) { return (k == 0 || k == s->L) ? 1 : s->R; }

static void mixed_radix_n(const shape_n_t* s, int64_t g, int64_t* dig) {
  for (int k = 0; k < s->L; ++k) {
    int64_t prod = 1;
    for (int j = k + 1; j < s->L; ++j) prod *= s->n[j];
    dig[k] = (g / prod) % s->n[k];
  }
}

static int64_t slice_len_n(const shape_n_t* s, int k) {
  return (int64_t)rank_n(s, k) * s->d[k] * rank_n(s, k + 1);
}

static const float* slice_n(const shape_n_t* s, const float* G, int k, int64_t t, int64_t i) {
  return G + (t * s->n[k] + i) * slice_len_n(s, k);
}

/* X[k] for k = 0..L-1 of one row; X[k] holds m_k * r_{k+1} doubles. */
static void chain_n(const shape_n_t* s, const float* const* G, int64_t t, const int64_t* dig, double** X) {
  const float* S0 = slice_n(s, G[0], 0, t, dig[0]);
  for (int64_t e = 0; e < slice_len_n(s, 0); ++e) X[0][e] = (double)S0[e];
  int64_t m = s->d[0];
  for (int k = 1; k < s->L; ++k) {
    const float* S = slice_n(s, G[k], k, t, dig[k]);
    int rk = rank_n(s, k);
    int64_t cols = (int64_t)s->d[k] * rank_n(s, k + 1);
    for (int64_t r = 0; r < m; ++r)
      for (int64_t c = 0; c < cols; ++c) {
        double acc = 0.0;
        for (int a = 0; a < rk; ++a) acc += X[k - 1][r * rk + a] * (double)S[a * cols + c];
        X[k][r * cols + c] = acc;
      }
    m *= s->d[k];
  }
}

static double** alloc_chain_n(const shape_n_t* s) {
  double** X = (double**)malloc(sizeof(double*) * s->L);
  int64_t m = 1;
  for (int k = 0; k < s->L; ++k) {
    m *= s->d[k];
    X[k] = (double*)malloc(sizeof(double) * m * rank_n(s, k + 1));
  }
  return X;
}

static void free_chain_n(const shape_n_t* s, double** X) {
  for (int k = 0; k < s->L; ++k) free(X[k]);
  free(X);
}

static int64_t dimD_n(const shape_n_t* s) {
  int64_t D = 1;
  for (int k = 0; k < s->L; ++k) D *= s->d[k];
  return D;
}

/* Forward with L cores: V [T*B][D] (sum pooling, empty bag = 0).  Returns the
 * number of invalid indices met. */
int64_t orc_forward_n(const shape_n_t* s, const float* const* G, const int64_t* idx, int64_t M,
                      const int64_t* offsets, double* V) {
  int64_t D = dimD_n(s), nb = (int64_t)s->T * s->B;
  double** X = alloc_chain_n(s);
  int64_t dig[ORC_MAXL];
  int64_t invalid = 0;
  (void)M;
  for (int64_t gb = 0; gb < nb; ++gb) {
    int64_t t = gb / s->B;
    int64_t lo = offsets ? offsets[gb] : gb, hi = offsets ? offsets[gb + 1] : gb + 1;
    double* out = V + gb * D;
    for (int64_t j = 0; j < D; ++j) out[j] = 0.0;
    for (int64_t o = lo; o < hi; ++o) {
      int64_t g = idx[o];
      if (g < 0 || g >= s->N) {
        ++invalid;
        continue;
      }
      mixed_radix_n(s, g, dig);
      chain_n(s, G, t, dig, X);
      for (int64_t j = 0; j < D; ++j) out[j] += X[s->L - 1][j];
    }
  }
  free_chain_n(s, X);
  return invalid;
}

/* Backward with L cores of L = sum <dV, V> into dense core gradients dG[k]
 * (doubles, shaped like core k, overwritten).  Per occurrence, with
 * dX_{L-1} = dV[bag] (the chain rule through the chain above):
 *   for k = L-1 .. 1:  dS_k += X_{k-1}^T dX_k     (dX_k viewed as m_{k-1} x d_k r_{k+1})
 *                      dX_{k-1} = dX_k S_k^T      (m_{k-1} x r_k)
 *   dS_0 += dX_0.
 * For L = 3: dG3 += C^T dE, dC = dE D^T, dG2 += A^T dC, dG1 += dC B^T (Eq. 1).
 * Optional want: NULL, or L masks (each NULL or per-slice flags [T*n_k]); when
 * some mask is given, an occurrence that touches no wanted slice of any core is
 * skipped, so only the wanted slices' gradients are guaranteed (those stay
 * exact: every occurrence that adds to them is kept, in the same order). */
int64_t orc_backward_n(const shape_n_t* s, const float* const* G, const int64_t* idx, int64_t M,
                       const int64_t* offsets, const float* dV, double* const* dG, const uint8_t* const* want) {
  int64_t D = dimD_n(s);
  for (int k = 0; k < s->L; ++k) memset(dG[k], 0, sizeof(double) * s->T * s->n[k] * slice_len_n(s, k));
  int64_t* bag = (int64_t*)malloc(sizeof(int64_t) * (M > 0 ? M : 1));
  if (!offsets) {
    for (int64_t o = 0; o < M; ++o) bag[o] = o;
  } else {
    for (int64_t gb = 0; gb < (int64_t)s->T * s->B; ++gb)
      for (int64_t o = offsets[gb]; o < offsets[gb + 1]; ++o) bag[o] = gb;
  }
  double** X = alloc_chain_n(s);
  double** dX = alloc_chain_n(s);
  int64_t dig[ORC_MAXL];
  int64_t invalid = 0;
  int masked = 0;  /* as in orc_backward: select only when some mask is given */
  for (int k = 0; want && k < s->L; ++k) masked |= want[k] != NULL;
  for (int64_t o = 0; o < M; ++o) {
    int64_t g = idx[o];
    if (g < 0 || g >= s->N) {
      ++invalid;
      continue;
    }
    int64_t gb = bag[o], t = gb / s->B;
    mixed_radix_n(s, g, dig);
    if (masked) {
      int w = 0;
      for (int k = 0; k < s->L && !w; ++k) w = want[k] && want[k][t * s->n[k] + dig[k]];
      if (!w) continue;
    }
    chain_n(s, G, t, dig, X);
    for (int64_t j = 0; j < D; ++j) dX[s->L - 1][j] = (double)dV[gb * D + j];
    int64_t m = D / s->d[s->L - 1];  /* m_{L-2} */
    for (int k = s->L - 1; k >= 1; --k) {
      const float* S = slice_n(s, G[k], k, t, dig[k]);
      int rk = rank_n(s, k);
      int64_t cols = (int64_t)s->d[k] * rank_n(s, k + 1);
      double* dS = dG[k] + (t * s->n[k] + dig[k]) * slice_len_n(s, k);
      for (int a = 0; a < rk; ++a)
        for (int64_t c = 0; c < cols; ++c) {
          double acc = 0.0;
          for (int64_t r = 0; r < m; ++r) acc += X[k - 1][r * rk + a] * dX[k][r * cols + c];
          dS[a * cols + c] += acc;
        }
      for (int64_t r = 0; r < m; ++r)
        for (int a = 0; a < rk; ++a) {
          double acc = 0.0;
          for (int64_t c = 0; c < cols; ++c) acc += dX[k][r * cols + c] * (double)S[a * cols + c];
          dX[k - 1][r * rk + a] = acc;
        }
      m /= s->d[k - 1];
    }
    double* dS0 = dG[0] + (t * s->n[0] + dig[0]) * slice_len_n(s, 0);
    for (int64_t e = 0; e < slice_len_n(s, 0); ++e) dS0[e] += dX[0][e];
  }
  free_chain_n(s, X);
  free_chain_n(s, dX);
  free(bag);
  return invalid;
}

/* Plain SGD step: out = G - lr * dG (no momentum, no weight decay). */
void orc_sgd(const float* G, const double* dG, int64_t count, double lr, double* out) {
  for (int64_t i = 0; i < count; ++i) out[i] = (double)G[i] - lr * dG[i];
}

/* Prefix-based index grouping of Section 3.3 (Fig. 4), as canonical integer
 * arrays: per table, sort the indices ascending, keep exact uniques, take the
 * mixed-radix digits, and run-length encode the (i1, i2) prefixes.
 *   uniq_t/uniq_g [U]  ascending (table, row) pairs
 *   inv [M]            rank of occurrence o's (table, row) in uniq, -1 if invalid
 *   occ_start [U+1]    occurrences of uniq[u] are occ_pos[occ_start[u] .. occ_start[u+1])
 *   occ_pos [nvalid]   positions stably sorted by (table, row, position)
 *   pg_start [P+1]     prefix group p covers uniq[pg_start[p] .. pg_start[p+1])
 *   pg_t/pg_q [P]      its table and prefix id q = i1*n2 + i2
 *   counts[3]          U, P, nvalid
 */
typedef struct {
  int64_t t, g, pos;
} occ_t;

static int cmp_occ(const void* x, const void* y) {
  const occ_t* a = (const occ_t*)x;
  const occ_t* b = (const occ_t*)y;
  if (a->t != b->t) return a->t < b->t ? -1 : 1;
  if (a->g != b->g) return a->g < b->g ? -1 : 1;
  if (a->pos != b->pos) return a->pos < b->pos ? -1 : 1;
  return 0;
}

void orc_grouping(const shape_t* s, const int64_t* idx, int64_t M, const int64_t* offsets, int64_t* uniq_t,
                  int64_t* uniq_g, int64_t* inv, int64_t* occ_start, int64_t* occ_pos, int64_t* pg_start,
                  int64_t* pg_t, int64_t* pg_q, int64_t counts[3]) {
  int64_t* bag = (int64_t*)malloc(sizeof(int64_t) * (M > 0 ? M : 1));
  bag_of_occurrences(s, M, offsets, bag);
  occ_t* v = (occ_t*)malloc(sizeof(occ_t) * (M > 0 ? M : 1));
  int64_t nv = 0;
  for (int64_t o = 0; o < M; ++o) {
    inv[o] = -1;
    if (idx[o] < 0 || idx[o] >= s->N) continue;
    v[nv].t = bag[o] / s->B;
    v[nv].g = idx[o];
    v[nv].pos = o;
    ++nv;
  }
  qsort(v, (size_t)nv, sizeof(occ_t), cmp_occ);
  int64_t U = 0, P = 0;
  int64_t last_pt = -1, last_pq = -1;
  for (int64_t i = 0; i < nv; ++i) {
    int new_row = (i == 0) || v[i].t != v[i - 1].t || v[i].g != v[i - 1].g;
    if (new_row) {
      int64_t dig[3];
      mixed_radix3(v[i].g, s->n, dig);
      int64_t q = dig[0] * s->n[1] + dig[1];
      if (v[i].t != last_pt || q != last_pq) {
        pg_start[P] = U;
        pg_t[P] = v[i].t;
        pg_q[P] = q;
        ++P;
        last_pt = v[i].t;
        last_pq = q;
      }
      uniq_t[U] = v[i].t;
      uniq_g[U] = v[i].g;
      occ_start[U] = i;
      ++U;
    }
    inv[v[i].pos] = U - 1;
    occ_pos[i] = v[i].pos;
  }
  occ_start[U] = nv;
  pg_start[P] = U;
  counts[0] = U;
  counts[1] = P;
  counts[2] = nv;
  free(v);
  free(bag);
}
