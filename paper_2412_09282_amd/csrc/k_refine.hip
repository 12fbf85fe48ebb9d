// Loss-driven refinement of a quantized layer (the QuantLoss / FineTuneCodebook / BeamSearchOptimize
// loop of Alg. 1), on the layer in reordered channel order.  With H = X^T X (the paper's X X^T for
// activations stored tokens x N) and R = W - W_hat:
//   QuantLoss = ||W X^T - W_hat X^T||^2 = sum_r R_r H R_r^T,  dQuantLoss / dW_hat = -2 R H.
//
// Kernels:
//  * gemm_f64_kernel: C = op(A) B in fp64 (H = X^T X from fp32 activations, G = R H), a 128 x 128
//    tile per workgroup, 8 x 8 outputs per thread, operands staged through LDS as fp64.
//  * row_dot_kernel: the per-row loss sum_j R_rj G_rj in a fixed order.
//  * code_sum_partial / code_sum_final: per-code sums of fp64 vectors (the codebook gradient), one
//    owner thread per code adding its members in vector order, then the block partials folded in
//    block order -- deterministic, no atomics.
//  * adam_kernel: one Adam step (moments in fp64, bias correction from the host) on an fp32 book.
//  * refine_group_kernel: the width-1 code search of one column group for every row, minimising
//    QuantLoss with all other codes fixed; the running product S = R H of the later columns is
//    updated by the chosen codeword change.  One wave per row, eight rows per workgroup.
#include "crvq_internal.h"

namespace crvq {
namespace {

constexpr int kGBM = 128, kGBN = 128, kGBK = 8;

template <typename T>
__device__ __forceinline__ double to_f64(T x) {
  return static_cast<double>(x);
}

// C[i][j] = sum_k opA(i, k) B(k, j) for i < M, j < Nc, k < Kd, where opA(i, k) = A[i * lda + k], or
// A[k * lda + i] when TRANS_A, and B(k, j) = B[k * ldb + j].  Products are formed in fp64 (exact for
// fp32 operands) and accumulated with fused multiply-adds in k order.
template <typename TA, typename TB, bool TRANS_A>
__global__ __launch_bounds__(256) void gemm_f64_kernel(int64_t M, int64_t Nc, int64_t Kd, const TA* __restrict__ A,
                                                       int64_t lda, const TB* __restrict__ B, int64_t ldb,
                                                       double* __restrict__ C, int64_t ldc) {
  __shared__ double As[kGBK][kGBM];
  __shared__ double Bs[kGBK][kGBN];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int64_t i0 = static_cast<int64_t>(blockIdx.y) * kGBM, j0 = static_cast<int64_t>(blockIdx.x) * kGBN;
  double acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0;
  for (int64_t k0 = 0; k0 < Kd; k0 += kGBK) {
#pragma unroll
    for (int s = 0; s < kGBM * kGBK / 256; ++s) {
      const int e = tid + 256 * s;
      int ii, kk;
      if (TRANS_A) {  // consecutive threads read consecutive i (contiguous in memory)
        ii = e % kGBM;
        kk = e / kGBM;
      } else {        // consecutive threads read consecutive k of one row
        kk = e % kGBK;
        ii = e / kGBK;
      }
      const int64_t gi = i0 + ii, gk = k0 + kk;
      double v = 0.0;
      if (gi < M && gk < Kd) v = to_f64(TRANS_A ? A[gk * lda + gi] : A[gi * lda + gk]);
      As[kk][ii] = v;
    }
#pragma unroll
    for (int s = 0; s < kGBN * kGBK / 256; ++s) {
      const int e = tid + 256 * s;
      const int jj = e % kGBN, kk = e / kGBN;
      const int64_t gj = j0 + jj, gk = k0 + kk;
      Bs[kk][jj] = (gj < Nc && gk < Kd) ? to_f64(B[gk * ldb + gj]) : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kGBK; ++kk) {
      double a[8], b[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 8; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t gi = i0 + ty + 16 * i;
    if (gi >= M) continue;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t gj = j0 + tx + 16 * j;
      if (gj < Nc) C[gi * ldc + gj] = acc[i][j];
    }
  }
}

// out[r] = sum_{j < n} A[r * lda + j] * B[r * ldb + j]: strided per-thread sums, then a fixed tree.
__global__ __launch_bounds__(256) void row_dot_kernel(int64_t n, const double* __restrict__ A, int64_t lda,
                                                      const double* __restrict__ B, int64_t ldb,
                                                      double* __restrict__ out) {
  __shared__ double red[256];
  const int64_t r = blockIdx.x;
  double acc = 0.0;
  for (int64_t j = threadIdx.x; j < n; j += 256) acc = acc + A[r * lda + j] * B[r * ldb + j];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w) red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[r] = red[0];
}

// ---- per-code sums ------------------------------------------------------------------------------
constexpr int kCsVec = 256;      // vectors staged per round
constexpr int kCsMaxOwn = 4;     // codes per thread (K <= 1024)

// Block b sums the vectors [b * per_block, ...) of a vector set over an fp64 matrix (vector
// v = r * vpr + g at element r * ld + g * d).  Thread t owns codes t, t + 256, ... and adds, in
// vector order, every staged vector whose code it owns.  part layout: [k * d + t][block].
__global__ __launch_bounds__(256) void code_sum_partial(const double* __restrict__ X, int64_t vpr, int64_t ld, int d,
                                                        int64_t n, const int32_t* __restrict__ codes, int K,
                                                        int64_t per_block, int64_t nblocks,
                                                        double* __restrict__ part, int* __restrict__ pcount) {
  __shared__ double sv[kCsVec * 16];
  __shared__ int sc[kCsVec];
  const int tid = threadIdx.x;
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per_block;
  const int64_t b1 = b0 + per_block < n ? b0 + per_block : n;
  double acc[kCsMaxOwn][16];
  int cnt[kCsMaxOwn];
#pragma unroll
  for (int j = 0; j < kCsMaxOwn; ++j) {
    cnt[j] = 0;
#pragma unroll
    for (int t = 0; t < 16; ++t) acc[j][t] = 0.0;
  }
  for (int64_t base = b0; base < b1; base += kCsVec) {
    const int rn = static_cast<int>(b1 - base < kCsVec ? b1 - base : kCsVec);
    for (int v = tid; v < rn; v += 256) {
      const int64_t i = base + v;
      const int64_t r = i / vpr, g = i - r * vpr;
      const double* p = X + r * ld + g * d;
      for (int t = 0; t < d; ++t) sv[v * d + t] = p[t];
      const int c = codes[i];
      sc[v] = (c >= 0 && c < K) ? c : -1;
    }
    __syncthreads();
    for (int v = 0; v < rn; ++v) {
      const int c = sc[v];
      if (c >= 0 && (c & 255) == tid) {
        const int j = c >> 8;
#pragma unroll
        for (int jj = 0; jj < kCsMaxOwn; ++jj) {
          if (jj == j) {
            ++cnt[jj];
#pragma unroll
            for (int t = 0; t < 16; ++t)
              if (t < d) acc[jj][t] = acc[jj][t] + sv[v * d + t];
          }
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < kCsMaxOwn; ++j) {
    const int k = tid + 256 * j;
    if (k >= K) continue;
#pragma unroll
    for (int t = 0; t < 16; ++t)
      if (t < d) part[(static_cast<int64_t>(k) * d + t) * nblocks + blockIdx.x] = acc[j][t];
    pcount[static_cast<int64_t>(k) * nblocks + blockIdx.x] = cnt[j];
  }
}

// One wave per sum element: lanes fold blocks lane, lane + 64, ... in order, then a fixed butterfly.
__global__ __launch_bounds__(256) void code_sum_final(const double* __restrict__ part, const int* __restrict__ pcount,
                                                      int64_t nblocks, int64_t K, int d, double* __restrict__ sums,
                                                      int32_t* __restrict__ counts) {
  const int lane = threadIdx.x & 63;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (e >= K * d) return;
  const int64_t k = e / d;
  const int t = static_cast<int>(e - k * d);
  double acc = 0.0;
  int cnt = 0;
  for (int64_t b = lane; b < nblocks; b += 64) {
    acc = acc + part[e * nblocks + b];
    cnt += pcount[k * nblocks + b];
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    acc = acc + __shfl_xor(acc, m);
    cnt += __shfl_xor(cnt, m);
  }
  if (lane == 0) {
    sums[e] = acc;
    if (counts && t == 0) counts[k] = cnt;
  }
}

// ---- Adam ---------------------------------------------------------------------------------------
// g = scale * grad; m = b1 m + (1 - b1) g; v = b2 v + (1 - b2) g^2; C -= lr * (m / bc1) / (sqrt(v / bc2) + eps)
// with the bias corrections bc1 = 1 - b1^t, bc2 = 1 - b2^t from the host; fp64 throughout, the
// codeword rounded once to fp32.  Each operation is rounded on its own (no contraction).
__global__ __launch_bounds__(256) void adam_kernel(int64_t n, float* __restrict__ C, const double* __restrict__ grad,
                                                   double scale, double* __restrict__ m, double* __restrict__ v,
                                                   double lr, double b1, double b2, double bc1, double bc2,
                                                   double eps) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n) return;
  const double g = scale * grad[i];
  const double mi = b1 * m[i] + (1.0 - b1) * g;
  const double vi = b2 * v[i] + (1.0 - b2) * (g * g);
  m[i] = mi;
  v[i] = vi;
  const double mh = mi / bc1;
  const double vh = vi / bc2;
  C[i] = static_cast<float>(static_cast<double>(C[i]) - lr * mh / (sqrt(vh) + eps));
}

// ---- width-1 code search of one column group ------------------------------------------------------
constexpr int kRfRows = 8;      // rows per workgroup, one wave each
constexpr int kRfThreads = 64 * kRfRows;
constexpr int kRfChunk = 4096;  // doubles of the H block staged per chunk (kRfChunk / d columns)

__device__ __forceinline__ double book_elem(const void* C, int type, int64_t i) {
  if (type == ET_F32) return static_cast<double>(static_cast<const float*>(C)[i]);
  return static_cast<double>(__uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(C)[i]) << 16));
}

// Group g (columns g*d .. g*d + d - 1) of rows blockIdx.x * 8 + wave.  With s = (R H)_g (held in S),
// the loss change of moving the code from c0 to c_k is
//   c_k^T Hgg c_k - 2 c_k . (s + Hgg c0) - (the same at c0),
// so the row takes the k minimising f(k) = a_k - 2 c_k . b with a_k = c_k^T Hgg c_k and
// b = s + Hgg c0 (lowest k on ties).  A moved row subtracts delta = c_k - c0 from its residual and
// delta^T H[g rows, c] from S[r, c] for the later columns c < n_cols.  A code outside [0, K) leaves the
// row unchanged.
template <int DMAX>
__global__ __launch_bounds__(kRfThreads) void refine_group_kernel(int64_t M, int d, int64_t g, int64_t n_cols,
                                                                 double* __restrict__ R, int64_t ldr,
                                                                 double* __restrict__ S, int64_t lds,
                                                                 const double* __restrict__ H, int64_t ldh,
                                                                 const void* __restrict__ Cb, int c_type, int K,
                                                                 int32_t* __restrict__ codes, int64_t ldq) {
  extern __shared__ double sm[];
  double* Cs = sm;             // K * d
  double* Ak = Cs + K * d;     // K
  double* Hg = Ak + K;         // d * d
  double* Hc = Hg + 256;       // kRfChunk
  __shared__ double s_delta[kRfRows][16];
  __shared__ double s_b[kRfRows][16];
  __shared__ int s_moved[kRfRows];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int64_t c0 = g * d;
  for (int e = tid; e < K * d; e += kRfThreads) Cs[e] = book_elem(Cb, c_type, e);
  for (int e = tid; e < d * d; e += kRfThreads) Hg[e] = H[(c0 + e / d) * ldh + c0 + e % d];
  __syncthreads();
  for (int k = tid; k < K; k += kRfThreads) {
    double a = 0.0;
    for (int t = 0; t < d; ++t) {
      double h = 0.0;
      for (int u = 0; u < d; ++u) h = h + Hg[t * d + u] * Cs[k * d + u];
      a = a + Cs[k * d + t] * h;
    }
    Ak[k] = a;
  }
  __syncthreads();
  const int64_t r = static_cast<int64_t>(blockIdx.x) * kRfRows + w;
  const int cur = r < M ? codes[r * ldq + g] : -1;
  const bool active = cur >= 0 && cur < K;
  if (active && lane < d) {  // b = s + Hgg c_cur, one lane per element
    double h = 0.0;
    for (int u = 0; u < d; ++u) h = h + Hg[lane * d + u] * Cs[cur * d + u];
    s_b[w][lane] = S[r * lds + c0 + lane] + h;
  }
  __syncthreads();
  int moved = 0;
  if (active) {
    double b[DMAX];
#pragma unroll
    for (int t = 0; t < DMAX; ++t) b[t] = t < d ? s_b[w][t] : 0.0;
    double best = __builtin_inf();
    int bk = K;
#pragma unroll 1
    for (int k = lane; k < K; k += 64) {
      double dot = 0.0;
#pragma unroll
      for (int t = 0; t < DMAX; ++t)
        if (t < d) dot = dot + Cs[k * d + t] * b[t];
      const double f = Ak[k] - 2.0 * dot;
      if (f < best) {
        best = f;
        bk = k;
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const double ob = __shfl_xor(best, m);
      const int ok = __shfl_xor(bk, m);
      if (ob < best || (ob == best && ok < bk)) {
        best = ob;
        bk = ok;
      }
    }
    if (bk < K && bk != cur) {
      moved = 1;
      if (lane < d) {
        const double delta = Cs[bk * d + lane] - Cs[cur * d + lane];
        s_delta[w][lane] = delta;
        R[r * ldr + c0 + lane] = R[r * ldr + c0 + lane] - delta;
      }
      if (lane == 0) codes[r * ldq + g] = bk;
    }
  }
  if (lane == 0) s_moved[w] = moved;
  __syncthreads();
  int any = 0;
  for (int i = 0; i < kRfRows; ++i) any |= s_moved[i];
  if (!any) return;  // the same for every thread of the block
  const int64_t cw = kRfChunk / d;  // columns per chunk
  for (int64_t cs = c0 + d; cs < n_cols; cs += cw) {
    const int64_t cn = n_cols - cs < cw ? n_cols - cs : cw;
    for (int64_t e = tid; e < d * cn; e += kRfThreads) {
      const int64_t t = e / cn, c = e - t * cn;
      Hc[t * cw + c] = H[(c0 + t) * ldh + cs + c];
    }
    __syncthreads();
    if (moved) {
      for (int64_t c = lane; c < cn; c += 64) {
        double acc = 0.0;
        for (int t = 0; t < d; ++t) acc = acc + s_delta[w][t] * Hc[t * cw + c];
        S[r * lds + cs + c] = S[r * lds + cs + c] - acc;
      }
    }
    __syncthreads();
  }
}

}  // namespace

// ---- launchers -----------------------------------------------------------------------------------
hipError_t launch_gemm_f64(int64_t M, int64_t Nc, int64_t Kd, const void* A, int a_type, bool trans_a, int64_t lda,
                           const void* B, int b_type, int64_t ldb, double* C, int64_t ldc, hipStream_t stream) {
  if (M <= 0 || Nc <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(cdiv(Nc, kGBN)), static_cast<unsigned>(cdiv(M, kGBM)));
#define CRVQ_GEMM(TA, TB, TR)                                                                              \
  hipLaunchKernelGGL((gemm_f64_kernel<TA, TB, TR>), grid, dim3(256), 0, stream, M, Nc, Kd,                 \
                     static_cast<const TA*>(A), lda, static_cast<const TB*>(B), ldb, C, ldc)
  if (a_type == ET_F32 && b_type == ET_F32) {
    if (trans_a) CRVQ_GEMM(float, float, true); else CRVQ_GEMM(float, float, false);
  } else if (a_type == ET_F64 && b_type == ET_F64) {
    if (trans_a) CRVQ_GEMM(double, double, true); else CRVQ_GEMM(double, double, false);
  } else {
    return hipErrorInvalidValue;
  }
#undef CRVQ_GEMM
  return hipGetLastError();
}

hipError_t launch_row_dot(int64_t M, int64_t n, const double* A, int64_t lda, const double* B, int64_t ldb,
                          double* out, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(row_dot_kernel, dim3(static_cast<unsigned>(M)), dim3(256), 0, stream, n, A, lda, B, ldb, out);
  return hipGetLastError();
}

static int64_t code_sum_blocks(int64_t n) {
  const int64_t rounds = cdiv(n > 0 ? n : 1, kCsVec);
  return rounds < 1024 ? rounds : 1024;
}

size_t code_sums_ws_bytes(int64_t n, int64_t K, int d) {
  WsCursor c(nullptr);
  const int64_t nb = code_sum_blocks(n);
  c.take<double>(static_cast<size_t>(nb * K * d));
  c.take<int>(static_cast<size_t>(nb * K));
  return c.used;
}

hipError_t launch_code_sums(const double* X, int64_t vpr, int64_t ld, int d, int64_t n, const int32_t* codes,
                            int64_t K, double* sums, int32_t* counts, void* ws, hipStream_t stream) {
  WsCursor cur(ws);
  int64_t nb = code_sum_blocks(n);
  const int64_t per_block = cdiv(cdiv(n > 0 ? n : 1, nb), kCsVec) * kCsVec;
  nb = cdiv(n > 0 ? n : 1, per_block);
  double* part = cur.take<double>(static_cast<size_t>(code_sum_blocks(n) * K * d));
  int* pcount = cur.take<int>(static_cast<size_t>(code_sum_blocks(n) * K));
  hipLaunchKernelGGL(code_sum_partial, dim3(static_cast<unsigned>(nb)), dim3(256), 0, stream, X, vpr, ld, d, n, codes,
                     static_cast<int>(K), per_block, nb, part, pcount);
  hipLaunchKernelGGL(code_sum_final, dim3(static_cast<unsigned>(cdiv(K * d, 4))), dim3(256), 0, stream, part, pcount,
                     nb, K, d, sums, counts);
  return hipGetLastError();
}

hipError_t launch_adam(int64_t n, float* C, const double* grad, double scale, double* m, double* v, double lr,
                       double b1, double b2, double bc1, double bc2, double eps, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(adam_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0, stream, n, C, grad, scale, m,
                     v, lr, b1, b2, bc1, bc2, eps);
  return hipGetLastError();
}

size_t refine_lds_bytes(int64_t K, int d) {
  return static_cast<size_t>(K * d + K + 256 + kRfChunk) * sizeof(double);
}

hipError_t launch_refine_book(int64_t M, int64_t N, int d, int64_t n_cols, double* R, int64_t ldr, const double* H,
                              int64_t ldh, const void* Cb, int c_type, int64_t K, int32_t* codes, int64_t ldq,
                              double* S, hipStream_t stream) {
  if (M <= 0 || n_cols <= 0) return hipSuccess;
  // S = R H[:, 0:n_cols]
  hipError_t e = launch_gemm_f64(M, n_cols, N, R, ET_F64, false, ldr, H, ET_F64, ldh, S, n_cols, stream);
  if (e != hipSuccess) return e;
  const size_t lds = refine_lds_bytes(K, d);
  const dim3 grid(static_cast<unsigned>(cdiv(M, kRfRows)));
  for (int64_t g = 0; g < n_cols / d; ++g) {
    if (d <= 8)
      hipLaunchKernelGGL(refine_group_kernel<8>, grid, dim3(kRfThreads), lds, stream, M, d, g, n_cols, R, ldr, S, n_cols,
                         H, ldh, Cb, c_type, static_cast<int>(K), codes, ldq);
    else
      hipLaunchKernelGGL(refine_group_kernel<16>, grid, dim3(kRfThreads), lds, stream, M, d, g, n_cols, R, ldr, S,
                         n_cols, H, ldh, Cb, c_type, static_cast<int>(K), codes, ldq);
  }
  return hipGetLastError();
}

}  // namespace crvq
