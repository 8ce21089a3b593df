// GPTQ in the transformed coordinates (eq. (7), Sec. III-F): the offline rounding of
// four-bit folded weights against the second moment G = Z Z^T of calibration tokens taken
// in the runtime transform's coordinates, with diagonal damping.  Four stages, each a few
// kernels:
//   transform: the prologue's transform alone (fold-before multiplier, unnormalized
//     blockwise butterfly in the prologue's stage order, fold-after multiplier), fp32
//     rows out; it gives the calibration tokens Z and the folded weight rows;
//   second moment: G = sum_t z_t z_t^T in fp64 (a register-tiled fp64 product);
//   factor: U upper triangular with (G + lambda I)^-1 = U^T U.  With the index reversal
//     P, the lower Cholesky factor L of A = P H P gives H = V V^T for the upper triangular
//     V = P L P, so U = V^-1 = P L^-1 P: a blocked Cholesky (64-wide diagonal blocks in
//     one wave's registers, row-parallel triangular solves, fp64 product updates of the
//     trailing matrix) and a triangular inverse that merges neighbouring diagonal blocks
//     level by level, so its large products run with many tiles;
//   sweep: the lazy-batch column sweep in fp64, 128 columns per block: inside a block the
//     columns are rounded one at a time for 4 rows per workgroup with the rows' block in
//     LDS; after the block one fp64 product pushes the block's errors onto the later
//     columns.  Every operation and its order follow the fp64 contract of the sweep, so the
//     codes are reproducible bit for bit.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fq_device.hpp"
#include "fq_launch.hpp"

namespace fq {

// ---------------------------------------------------------------------------------------
// transform

// One workgroup of E threads per E consecutive channels of a row (E = max(b, 128); K is
// a multiple of 128 and of b; grid x = rows, y = channel groups).  Stage h exchanges through LDS: the lower index of a pair
// gets a + c, the upper a - c, the same fp32 additions as the prologue's butterfly.
template <typename Tin, int E>
__global__ __launch_bounds__(E) void transform_kernel(const void *x, int64_t ldx, const float *pre,
                                                      const float *post, int K, int b, float *z) {
  __shared__ float buf[E];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const int c = blockIdx.y * E + t;
  float v;
  if constexpr (sizeof(Tin) == 2)
    v = bf16_lo(reinterpret_cast<const uint16_t *>(x)[row * ldx + c]);
  else
    v = reinterpret_cast<const float *>(x)[row * ldx + c];
  if (pre) v = v * pre[c];
  for (int h = 1; h < b; h *= 2) {
    buf[t] = v;
    __syncthreads();
    const float p = buf[t ^ h];
    v = (t & h) ? p - v : v + p;
    __syncthreads();
  }
  if (post) v = v * post[c];
  z[row * K + c] = v;
}

template <typename Tin>
static hipError_t launch_transform_t(const void *x, int64_t ldx, const float *pre, const float *post, int64_t M,
                                     int K, int b, float *z, hipStream_t s) {
  if (b <= 128) {
    hipLaunchKernelGGL((transform_kernel<Tin, 128>), dim3((unsigned)M, (unsigned)(K / 128)), dim3(128), 0, s, x,
                       ldx, pre, post, K, b, z);
  } else {
    hipLaunchKernelGGL((transform_kernel<Tin, 256>), dim3((unsigned)M, (unsigned)(K / 256)), dim3(256), 0, s, x,
                       ldx, pre, post, K, b, z);
  }
  return hipGetLastError();
}

hipError_t launch_transform(const void *x, bool x_is_f32, int64_t ldx, const float *pre, const float *post,
                            int64_t M, int K, int b, float *z, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (M > 2147483647) return hipErrorInvalidValue;
  return x_is_f32 ? launch_transform_t<float>(x, ldx, pre, post, M, K, b, z, s)
                  : launch_transform_t<uint16_t>(x, ldx, pre, post, M, K, b, z, s);
}

// ---------------------------------------------------------------------------------------
// fp64 product update: C (op)= sum_k A[i][k] B[k][j], every element's sum an fma chain in
// ascending k from +0, then C = C - sum, C = C + sum, C = -sum or C = sum.  64 x 64 tiles,
// 4 x 4 per thread, k in chunks of 16 through LDS.  A and B are addressed through element
// strides, so transposed operands need no copy.  `lower` computes only tiles on or below
// the diagonal and writes elements with i >= j; `mirror` also writes C[j][i].

enum : int { kSub = 0, kAdd = 1, kSetNeg = 2, kSet = 3 };

struct DProd {
  const void *a;
  int64_t a_si, a_sk;  // element strides of A: rows i, k
  const void *b;
  int64_t b_sk, b_sj;  // element strides of B: k, columns j
  double *c;
  int64_t ldc;
  int64_t m, n, kd;
  int mode;
  int lower, mirror;
  int kskip;  // B is lower triangular: tile column j0 sums k >= j0 only (the rest are zeros)
  int klow;   // A is lower triangular: tile row i0 sums k < i0 + 64 only
};

template <typename TA, typename TB>
__global__ __launch_bounds__(256) void dprod_kernel(DProd p) {
  constexpr int T = 64, KC = 16;
  __shared__ double as[KC][T + 1];
  __shared__ double bs[KC][T + 1];
  const int ti = blockIdx.y, tj = blockIdx.x;
  if ((p.lower || p.mirror) && tj > ti) return;
  const int tid = threadIdx.x;
  const int ty = tid / 16, tx = tid % 16;
  const int64_t i0 = (int64_t)ti * T, j0 = (int64_t)tj * T;
  const TA *A = reinterpret_cast<const TA *>(p.a);
  const TB *Bm = reinterpret_cast<const TB *>(p.b);
  double acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.0;
  const bool a_krun = p.a_sk == 1;  // consecutive lanes along k when k is the contiguous index
  const bool b_jrun = p.b_sj == 1;
  const int64_t kend = p.klow && i0 + T < p.kd ? i0 + T : p.kd;
  for (int64_t k0 = p.kskip ? j0 : 0; k0 < kend; k0 += KC) {
    __syncthreads();
#pragma unroll
    for (int u = 0; u < (T * KC) / 256; ++u) {
      const int e = tid + 256 * u;
      const int ii = a_krun ? e / KC : e % T, kk = a_krun ? e % KC : e / T;
      const int64_t gi = i0 + ii, gk = k0 + kk;
      as[kk][ii] = (gi < p.m && gk < p.kd) ? (double)A[gi * p.a_si + gk * p.a_sk] : 0.0;
      const int jj = b_jrun ? e % T : e / KC, kb = b_jrun ? e / T : e % KC;
      const int64_t gj = j0 + jj, gkb = k0 + kb;
      bs[kb][jj] = (gj < p.n && gkb < p.kd) ? (double)Bm[gkb * p.b_sk + gj * p.b_sj] : 0.0;
    }
    __syncthreads();
    const int kn = (int)(kend - k0 < KC ? kend - k0 : KC);
    for (int k = 0; k < kn; ++k) {
      double av[4], bv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) av[r] = as[k][ty * 4 + r];
#pragma unroll
      for (int c = 0; c < 4; ++c) bv[c] = bs[k][tx * 4 + c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = __builtin_fma(av[r], bv[c], acc[r][c]);
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t gi = i0 + ty * 4 + r;
    if (gi >= p.m) continue;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t gj = j0 + tx * 4 + c;
      if (gj >= p.n || (p.lower && gj > gi) || (p.mirror && gj > gi)) continue;
      double *dst = p.c + gi * p.ldc + gj;
      double v;
      switch (p.mode) {
        case kSub: v = *dst - acc[r][c]; break;
        case kAdd: v = *dst + acc[r][c]; break;
        case kSetNeg: v = -acc[r][c]; break;
        default: v = acc[r][c]; break;
      }
      *dst = v;
      if (p.mirror && gj != gi) p.c[gj * p.ldc + gi] = v;
    }
  }
}

template <typename TA, typename TB>
static hipError_t dprod(const DProd &p, hipStream_t s) {
  if (p.m <= 0 || p.n <= 0) return hipSuccess;
  const int64_t tm = (p.m + 63) / 64, tn = (p.n + 63) / 64;
  if (tm > 65535 || tn > 2147483647) return hipErrorInvalidValue;
  hipLaunchKernelGGL((dprod_kernel<TA, TB>), dim3((unsigned)tn, (unsigned)tm), dim3(256), 0, s, p);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void fill_kernel(double *d, int64_t n, double v) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < n) d[e] = v;
}

hipError_t launch_gptq_hessian(const float *z, int64_t ldz, int64_t T, int K, double *G, bool accumulate,
                               hipStream_t s) {
  if (T <= 0) {
    if (accumulate) return hipSuccess;
    const int64_t n = (int64_t)K * K;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, G, n, 0.0);
    return hipGetLastError();
  }
  // G[i][j] (+)= sum_t z[t][i] z[t][j]: A[i][t] = z[t][i], B[t][j] = z[t][j]; lower tiles,
  // mirrored
  DProd p{};
  p.a = z;
  p.a_si = 1;
  p.a_sk = ldz;
  p.b = z;
  p.b_sk = ldz;
  p.b_sj = 1;
  p.c = G;
  p.ldc = K;
  p.m = K;
  p.n = K;
  p.kd = T;
  p.mode = accumulate ? kAdd : kSet;
  p.mirror = 1;
  return dprod<float, float>(p, s);
}

// ---------------------------------------------------------------------------------------
// factor

// lambda = damp * mean(diag G), one workgroup; an all-zero diagonal gives lambda = 0,
// which the reversal kernel turns into the identity.
__global__ __launch_bounds__(256) void damp_kernel(const double *G, int K, double damp, double *lam) {
  __shared__ double part[256];
  double acc = 0.0;
  for (int i = threadIdx.x; i < K; i += 256) acc += G[(int64_t)i * K + i];
  part[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) lam[0] = damp * (part[0] / (double)K);
}

// A = P (G + lambda I) P (index reversal), or the identity when lambda = 0; X = 0.
__global__ __launch_bounds__(256) void reverse_kernel(const double *G, int K, const double *lam, double *A,
                                                      double *X) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)K * K) return;
  const int64_t i = e / K, j = e % K;
  const double l = lam[0];
  double v;
  if (l == 0.0)
    v = i == j ? 1.0 : 0.0;
  else
    v = G[(K - 1 - i) * (int64_t)K + (K - 1 - j)] + (i == j ? l : 0.0);
  A[e] = v;
  X[e] = 0.0;
}

constexpr int kNb = 64;  // Cholesky / inverse block

// The three small dense kernels of the factor run one wave per 64 x 64 block, each lane
// holding one row (or column) of 64 doubles in registers, every loop fully unrolled so the
// register indices are static; the entries other lanes need go through LDS.

// Cholesky of the diagonal block at k0 (lower), right-looking: lane i holds row i.  At step
// j every lane publishes its entry j, reads the pivot d = sqrt(l_jj) and 1/d, and takes
// column j's scaled entries l_cj = l_cj * (1/d) from LDS (the same product its owner forms),
// then updates its entries j < c <= i.  Selects, no divergent branches.  The block's upper
// part is written as zeros.
__global__ __launch_bounds__(64) void potrf_block_kernel(double *A, int K, int k0) {
  __shared__ double col[kNb];
  const int i = threadIdx.x;
  double r[kNb];
  const double *src = A + (int64_t)(k0 + i) * K + k0;
#pragma unroll
  for (int c = 0; c < kNb; ++c) r[c] = src[c];
#pragma unroll
  for (int j = 0; j < kNb; ++j) {
    col[i] = r[j];
    __syncthreads();
    const double d = sqrt(col[j]);
    const double inv = 1.0 / d;
    r[j] = i > j ? r[j] * inv : (i == j ? d : r[j]);
#pragma unroll
    for (int c = j + 1; c < kNb; ++c) {
      const double lc = col[c] * inv;
      r[c] = c <= i ? r[c] - r[j] * lc : r[c];
      if ((c & 7) == 7) __builtin_amdgcn_sched_barrier(0);  // few LDS values live at a time
    }
    __syncthreads();
  }
  double *dst = A + (int64_t)(k0 + i) * K + k0;
#pragma unroll
  for (int c = 0; c < kNb; ++c) dst[c] = c <= i ? r[c] : 0.0;
}

// Rows i >= k0 + 64 of the panel: x L_kk^T = a, one lane per row (64 per workgroup), the
// row in registers: x_c = x_c / l_cc, then x_c' -= x_c l_c'c for the later c' (each entry's
// subtractions in ascending c, the same arithmetic as the dot-product form).
__global__ __launch_bounds__(64) void trsm_rows_kernel(double *A, int K, int k0) {
  __shared__ double l[kNb][kNb];  // read at wave-uniform indices only
  const int tid = threadIdx.x;
  for (int e = tid; e < kNb * kNb; e += 64) l[e / kNb][e % kNb] = A[(int64_t)(k0 + e / kNb) * K + k0 + e % kNb];
  const int64_t row = (int64_t)k0 + kNb + (int64_t)blockIdx.x * 64 + tid;
  const int64_t rr = row < K ? row : K - 1;  // lanes past the end solve a copy of the last row, unstored
  double x[kNb];
#pragma unroll
  for (int c = 0; c < kNb; ++c) x[c] = A[rr * K + k0 + c];
  __syncthreads();
#pragma unroll
  for (int c = 0; c < kNb; ++c) {
    x[c] = x[c] / l[c][c];
#pragma unroll
    for (int c2 = c + 1; c2 < kNb; ++c2) x[c2] = x[c2] - x[c] * l[c2][c];
  }
  if (row < K)
#pragma unroll
    for (int c = 0; c < kNb; ++c) A[row * K + k0 + c] = x[c];
}

// X_ii = L_ii^-1 for every diagonal block (grid = K / 64): lane c computes column c,
// x = e_c, then x_m = x_m / l_mm and x_r -= l_rm x_m for r > m, m ascending.
__global__ __launch_bounds__(64) void triinv_block_kernel(const double *A, int K, double *X) {
  __shared__ double l[kNb][kNb];  // read at wave-uniform indices only
  const int c = threadIdx.x;
  const int k0 = blockIdx.x * kNb;
  for (int e = c; e < kNb * kNb; e += 64) l[e / kNb][e % kNb] = A[(int64_t)(k0 + e / kNb) * K + k0 + e % kNb];
  __syncthreads();
  double x[kNb];
#pragma unroll
  for (int r = 0; r < kNb; ++r) x[r] = r == c ? 1.0 : 0.0;
#pragma unroll
  for (int m = 0; m < kNb; ++m) {
    x[m] = x[m] / l[m][m];
#pragma unroll
    for (int r = m + 1; r < kNb; ++r) x[r] = x[r] - l[r][m] * x[m];
  }
#pragma unroll
  for (int r = 0; r < kNb; ++r) X[(int64_t)(k0 + r) * K + k0 + c] = x[r];
}

// U[i][j] = X[K-1-i][K-1-j] on and above the diagonal, 0 below.
__global__ __launch_bounds__(256) void unreverse_kernel(const double *X, int K, double *U) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)K * K) return;
  const int64_t i = e / K, j = e % K;
  U[e] = j >= i ? X[(K - 1 - i) * (int64_t)K + (K - 1 - j)] : 0.0;
}

size_t gptq_factor_ws_bytes(int K) {
  return ((size_t)2 * K * K + (size_t)(K / 2) * (K / 2)) * sizeof(double) + 256;
}

hipError_t launch_gptq_factor(const double *G, int K, double damp, double *U, void *ws, hipStream_t s) {
  double *A = static_cast<double *>(ws);
  double *X = A + (size_t)K * K;
  double *Tm = X + (size_t)K * K;  // B X_A of the inverse's merges, at most (K/2) x (K/2)
  double *lam = Tm + (size_t)(K / 2) * (K / 2);
  const int64_t n = (int64_t)K * K;
  const unsigned ge = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(damp_kernel, dim3(1), dim3(256), 0, s, G, K, damp, lam);
  hipLaunchKernelGGL(reverse_kernel, dim3(ge), dim3(256), 0, s, G, K, lam, A, X);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // blocked Cholesky, lower: A = L L^T in place
  for (int k0 = 0; k0 < K; k0 += kNb) {
    hipLaunchKernelGGL(potrf_block_kernel, dim3(1), dim3(64), 0, s, A, K, k0);
    const int rest = K - k0 - kNb;
    if (rest > 0) {
      hipLaunchKernelGGL(trsm_rows_kernel, dim3((unsigned)((rest + 63) / 64)), dim3(64), 0, s, A, K, k0);
      DProd p{};
      p.a = A + (int64_t)(k0 + kNb) * K + k0;  // L[i][k0 + k]
      p.a_si = K;
      p.a_sk = 1;
      p.b = A + (int64_t)(k0 + kNb) * K + k0;  // B[k][j] = L[j][k0 + k]
      p.b_sk = 1;
      p.b_sj = K;
      p.c = A + (int64_t)(k0 + kNb) * K + k0 + kNb;
      p.ldc = K;
      p.m = rest;
      p.n = rest;
      p.kd = kNb;
      p.mode = kSub;
      p.lower = 1;
      if ((e = dprod<double, double>(p, s)) != hipSuccess) return e;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // X = L^-1: the 64-wide diagonal blocks' inverses, then pairs of neighbouring diagonal
  // blocks merged level by level (widths 64, 128, 256, ...): for A = block 2t, C = block
  // 2t + 1 (possibly narrower at the end) and B the part of L below A and left of C,
  // X[C, A] = -X_C (B X_A).  Both products skip the zeros of their triangular operand.
  hipLaunchKernelGGL(triinv_block_kernel, dim3((unsigned)(K / kNb)), dim3(64), 0, s, A, K, X);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  for (int n = kNb; n < K; n *= 2) {
    for (int o = 0; o + n < K; o += 2 * n) {
      const int n2 = o + 2 * n <= K ? n : K - o - n;  // width of C
      DProd p{};
      p.a = A + (int64_t)(o + n) * K + o;  // B[r][k] = L[o + n + r][o + k]
      p.a_si = K;
      p.a_sk = 1;
      p.b = X + (int64_t)o * K + o;  // X_A[k][j]
      p.b_sk = K;
      p.b_sj = 1;
      p.c = Tm;
      p.ldc = n;
      p.m = n2;
      p.n = n;
      p.kd = n;
      p.mode = kSet;
      p.kskip = 1;
      if ((e = dprod<double, double>(p, s)) != hipSuccess) return e;
      DProd q{};
      q.a = X + (int64_t)(o + n) * K + o + n;  // X_C[r][k]
      q.a_si = K;
      q.a_sk = 1;
      q.b = Tm;  // Tm[k][j]
      q.b_sk = n;
      q.b_sj = 1;
      q.c = X + (int64_t)(o + n) * K + o;
      q.ldc = K;
      q.m = n2;
      q.n = n;
      q.kd = n2;
      q.mode = kSetNeg;
      q.klow = 1;
      if ((e = dprod<double, double>(q, s)) != hipSuccess) return e;
    }
  }
  hipLaunchKernelGGL(unreverse_kernel, dim3(ge), dim3(256), 0, s, X, K, U);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// sweep

constexpr int kSweepBlk = 128;  // columns per lazy batch
constexpr int kSweepRows = 4;   // rows per in-block workgroup (the column steps are latency-bound: more workgroups)

// Per row: A = max |w| (fp32, exact), the fp32 scale, fp64 inv = q / A and step = A / q,
// and the fp64 working copy.  One workgroup per row.
__global__ __launch_bounds__(256) void sweep_init_kernel(const float *w, int64_t ldw, int K, int bits,
                                                         float scale_mult, float *scales, double *rowp,
                                                         double *w64) {
  __shared__ float red[256];
  const int64_t row = blockIdx.x;
  const float *src = w + row * ldw;
  float a = 0.0f;
  for (int c = threadIdx.x; c < K; c += 256) {
    a = fmaxf(a, fabsf(src[c]));
    w64[row * K + c] = (double)src[c];
  }
  red[threadIdx.x] = a;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if ((int)threadIdx.x < h) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + h]);
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float A = red[0];
    const int q = (1 << (bits - 1)) - 1;
    scales[row] = A == 0.0f ? 0.0f : (A * scale_mult) / (float)q;
    rowp[2 * row] = A == 0.0f ? 0.0 : (double)q / (double)A;
    rowp[2 * row + 1] = (double)A / (double)q;
  }
}

// Columns [i1, i1 + 128) of 4 rows, one at a time: code, error, and the error pushed onto
// the block's later columns; the errors go to e [N, 128] for the product update.
__global__ __launch_bounds__(128) void sweep_block_kernel(const double *U, int64_t N, int K, int bits, int i1,
                                                          const double *rowp, double *w64, int8_t *codes,
                                                          double *e) {
  __shared__ double wb[kSweepRows][kSweepBlk + 1];
  __shared__ double es[kSweepRows];
  const int tid = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kSweepRows;
  const double q = (double)((1 << (bits - 1)) - 1);
  for (int x = tid; x < kSweepRows * kSweepBlk; x += 128) {
    const int r = x / kSweepBlk, c = x % kSweepBlk;
    wb[r][c] = r0 + r < N ? w64[(r0 + r) * K + i1 + c] : 0.0;
  }
  __syncthreads();
  for (int c = 0; c < kSweepBlk; ++c) {
    const int64_t gc = i1 + c;
    if (tid < kSweepRows) {
      const int64_t row = r0 + tid;
      double err = 0.0;
      if (row < N) {
        const double inv = rowp[2 * row], step = rowp[2 * row + 1];
        double k = 0.0;
        if (inv != 0.0) {  // a zero row keeps codes 0 and pushes no error
          k = rint(wb[tid][c] * inv);
          if (k > q) k = q;
          if (k < -q) k = -q;
          err = (wb[tid][c] - k * step) / U[gc * K + gc];
        }
        codes[row * K + gc] = (int8_t)k;
        e[row * kSweepBlk + c] = err;
      }
      es[tid] = err;
    }
    __syncthreads();
    const int rem = kSweepBlk - 1 - c;
    for (int x = tid; x < kSweepRows * rem; x += 128) {
      const int r = x / rem, c2 = c + 1 + x % rem;
      wb[r][c2] = __builtin_fma(-es[r], U[gc * K + i1 + c2], wb[r][c2]);
    }
    __syncthreads();
  }
}

size_t gptq_sweep_ws_bytes(int64_t N, int K) {
  return (size_t)N * K * sizeof(double) + (size_t)N * kSweepBlk * sizeof(double) + (size_t)N * 2 * sizeof(double) +
         256;
}

hipError_t launch_gptq_sweep(const float *w, int64_t ldw, const double *U, int64_t N, int K, int bits,
                             float scale_mult, int8_t *codes, float *scales, void *ws, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (N > 2147483647) return hipErrorInvalidValue;
  double *w64 = static_cast<double *>(ws);
  double *e = w64 + (size_t)N * K;
  double *rowp = e + (size_t)N * kSweepBlk;
  hipLaunchKernelGGL(sweep_init_kernel, dim3((unsigned)N), dim3(256), 0, s, w, ldw, K, bits, scale_mult, scales,
                     rowp, w64);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const unsigned gb = (unsigned)((N + kSweepRows - 1) / kSweepRows);
  for (int i1 = 0; i1 < K; i1 += kSweepBlk) {
    hipLaunchKernelGGL(sweep_block_kernel, dim3(gb), dim3(128), 0, s, U, N, K, bits, i1, rowp, w64, codes, e);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    const int i2 = i1 + kSweepBlk;
    if (i2 < K) {
      // w64[:, i2:] -= e U[i1:i2, i2:], each element's sum an fma chain in ascending k
      DProd p{};
      p.a = e;
      p.a_si = kSweepBlk;
      p.a_sk = 1;
      p.b = U + (int64_t)i1 * K + i2;
      p.b_sk = K;
      p.b_sj = 1;
      p.c = w64 + i2;
      p.ldc = K;
      p.m = N;
      p.n = K - i2;
      p.kd = kSweepBlk;
      p.mode = kSub;
      if ((err = dprod<double, double>(p, s)) != hipSuccess) return err;
    }
  }
  return hipSuccess;
}

}  // namespace fq
