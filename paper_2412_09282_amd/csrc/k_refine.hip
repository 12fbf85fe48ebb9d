// Loss-driven refinement of a quantized layer (the QuantLoss / FineTuneCodebook / BeamSearchOptimize
// loop of Alg. 1), on the layer in reordered channel order.  With H = X^T X (the paper's X X^T for
// activations stored tokens x N) and R = W - W_hat:
//   QuantLoss = ||W X^T - W_hat X^T||^2 = sum_r R_r H R_r^T,  dQuantLoss / dW_hat = -2 R H.
//
// Kernels:
//  * gemm_f64_kernel: C = op(A) B in fp64 (H = X^T X from fp32 activations, G = R H), a 128 x 128
//    tile per workgroup, 8 x 8 outputs per thread, operands staged through LDS as fp64.
//  * row_dot_kernel: the per-row loss sum_j R_rj G_rj in a fixed order.
//  * code_sum_wave_partial (K <= 256, d <= 8) or code_sum_partial, then code_sum_final: per-code sums
//    of fp64 vectors (the codebook gradient) in a fixed order -- per-wave LDS tables filled by ballot
//    peer groups, or one owner thread per code -- with the block partials folded in block order;
//    deterministic, no atomics.
//  * adam_kernel: one Adam step (moments in fp64, bias correction from the host) on an fp32 book.
//  * refine_block_kernel: the width-1 code search over a block of column groups (64 columns) for
//    every row, minimising QuantLoss with all other codes fixed; the running product S = R H is
//    updated in LDS inside the block and, for the later columns, by one product D H per block (D the
//    block's codeword changes).  One wave per row, eight rows per workgroup.
#include "crvq_internal.h"

namespace crvq {
namespace {

constexpr int kGBM = 128, kGBN = 128, kGBK = 8;
#ifndef CRVQ_GEMM_MFMA
#define CRVQ_GEMM_MFMA 1  // fp64 products without transpose on the matrix cores
#endif

template <typename T>
__device__ __forceinline__ double to_f64(T x) {
  return static_cast<double>(x);
}

// C[i][j] = sum_k opA(i, k) B(k, j) (or C[i][j] - that sum when SUB) for i < M, j < Nc, k < Kd, where
// opA(i, k) = A[i * lda + k], or A[k * lda + i] when TRANS_A, and B(k, j) = B[k * ldb + j].  Products are formed in fp64 (exact for
// fp32 operands) and accumulated with fused multiply-adds in k order.
template <typename TA, typename TB, bool TRANS_A, bool SUB>
__global__ __launch_bounds__(256) void gemm_f64_kernel(int64_t M, int64_t Nc, int64_t Kd, const TA* __restrict__ A,
                                                       int64_t lda, const TB* __restrict__ B, int64_t ldb,
                                                       double* __restrict__ C, int64_t ldc, int64_t kchunk,
                                                       int64_t c_part) {
  __shared__ double As[kGBK][kGBM];
  __shared__ double Bs[kGBK][kGBN];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int64_t i0 = static_cast<int64_t>(blockIdx.y) * kGBM, j0 = static_cast<int64_t>(blockIdx.x) * kGBN;
  // split over k: part blockIdx.z takes k in [kb, ke) and writes its own slice of C
  const int64_t kb = static_cast<int64_t>(blockIdx.z) * kchunk;
  const int64_t ke = kb + kchunk < Kd ? kb + kchunk : Kd;
  C += static_cast<int64_t>(blockIdx.z) * c_part;
  double acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0;
  for (int64_t k0 = kb; k0 < ke; k0 += kGBK) {
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
      if (gi < M && gk < ke) v = to_f64(TRANS_A ? A[gk * lda + gi] : A[gi * lda + gk]);
      As[kk][ii] = v;
    }
#pragma unroll
    for (int s = 0; s < kGBN * kGBK / 256; ++s) {
      const int e = tid + 256 * s;
      const int jj = e % kGBN, kk = e / kGBN;
      const int64_t gj = j0 + jj, gk = k0 + kk;
      Bs[kk][jj] = (gj < Nc && gk < ke) ? to_f64(B[gk * ldb + gj]) : 0.0;
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
      if (gj < Nc) C[gi * ldc + gj] = SUB ? C[gi * ldc + gj] - acc[i][j] : acc[i][j];
    }
  }
}

// The same product for fp64 A (row-major, not transposed) and B on the matrix cores: a 32 MW x 32 MW
// tile of C per workgroup, 16 MW x 16 MW per wave as MW x MW v_mfma_f64_16x16x4f64 tiles (MW = 4 for
// the long products, 2 for the short-k updates of the code search, which need more workgroups in
// flight to hide their loads), k staged through
// LDS 16 at a time (k-major, so the 16 lanes of an operand group read consecutive doubles).  Lane l
// of an MFMA supplies A[i0 + l % 16][k + l / 16] and B[k + l / 16][j0 + l % 16] and holds
// C[i0 + l / 16 + 4 r][j0 + l % 16], r < 4.  Each element is an fp64 dot product over its k range
// (the matrix core's accumulation within a group of 4, then k order).
constexpr int kMT = 128;  // C tile per workgroup and dimension of the long products (MW = 4)
constexpr int kMK = 16;   // k per LDS stage
typedef double d4v __attribute__((ext_vector_type(4)));
template <bool SUB, int kMW, typename TA = double, typename TB = double, bool TRANS_A = false>
__global__ __launch_bounds__(256) void gemm_f64_mfma_kernel(int64_t M, int64_t Nc, int64_t Kd, const TA* __restrict__ A,
                                                            int64_t lda, const TB* __restrict__ B, int64_t ldb,
                                                            double* __restrict__ C, int64_t ldc, int64_t kchunk,
                                                            int64_t c_part) {
  constexpr int kMT = 2 * 16 * kMW;  // C tile per workgroup and dimension (2 x 2 waves)
  __shared__ double As[kMK][kMT + 2];
  __shared__ double Bs[kMK][kMT + 2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wi = (wave >> 1) * 16 * kMW, wj = (wave & 1) * 16 * kMW;
  const int li = lane & 15, lk = lane >> 4;
  const int64_t i0 = static_cast<int64_t>(blockIdx.y) * kMT, j0 = static_cast<int64_t>(blockIdx.x) * kMT;
  const int64_t kb = static_cast<int64_t>(blockIdx.z) * kchunk;
  const int64_t ke = kb + kchunk < Kd ? kb + kchunk : Kd;
  C += static_cast<int64_t>(blockIdx.z) * c_part;
  d4v acc[kMW][kMW];
#pragma unroll
  for (int a = 0; a < kMW; ++a)
#pragma unroll
    for (int b = 0; b < kMW; ++b) acc[a][b] = d4v{0.0, 0.0, 0.0, 0.0};
  // stage k0's operands are read into registers one stage ahead, so their loads overlap the MFMAs
  constexpr int kL = kMT * kMK / 256;
  double pa[kL], pb[kL];
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int s = 0; s < kL; ++s) {
      const int e = tid + 256 * s;
      // consecutive threads: consecutive k of one row of A, or consecutive i of one row of A^T
      const int kk = TRANS_A ? e / kMT : e % kMK, ii = TRANS_A ? e % kMT : e / kMK;
      const int64_t gi = i0 + ii, gk = k0 + kk;
      pa[s] = (gi < M && gk < ke) ? to_f64(TRANS_A ? A[gk * lda + gi] : A[gi * lda + gk]) : 0.0;
      const int jj = e % kMT, kb2 = e / kMT;  // consecutive threads: consecutive j of one row of B
      const int64_t gj = j0 + jj, gk2 = k0 + kb2;
      pb[s] = (gj < Nc && gk2 < ke) ? to_f64(B[gk2 * ldb + gj]) : 0.0;
    }
  };
  if (kb < ke) fetch(kb);
  for (int64_t k0 = kb; k0 < ke; k0 += kMK) {
#pragma unroll
    for (int s = 0; s < kL; ++s) {
      const int e = tid + 256 * s;
      if (TRANS_A)
        As[e / kMT][e % kMT] = pa[s];
      else
        As[e % kMK][e / kMK] = pa[s];
      Bs[e / kMT][e % kMT] = pb[s];
    }
    __syncthreads();
    if (k0 + kMK < ke) fetch(k0 + kMK);
#pragma unroll
    for (int ks = 0; ks < kMK; ks += 4) {
      double a[kMW], b[kMW];
#pragma unroll
      for (int t = 0; t < kMW; ++t) {
        a[t] = As[ks + lk][wi + 16 * t + li];
        b[t] = Bs[ks + lk][wj + 16 * t + li];
      }
#pragma unroll
      for (int ta = 0; ta < kMW; ++ta)
#pragma unroll
        for (int tb = 0; tb < kMW; ++tb)
          acc[ta][tb] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[ta], b[tb], acc[ta][tb], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int ta = 0; ta < kMW; ++ta)
#pragma unroll
    for (int tb = 0; tb < kMW; ++tb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gi = i0 + wi + 16 * ta + lk + 4 * r, gj = j0 + wj + 16 * tb + li;
        if (gi < M && gj < Nc) C[gi * ldc + gj] = SUB ? C[gi * ldc + gj] - acc[ta][tb][r] : acc[ta][tb][r];
      }
}

// C[i][j] = sum over parts p = 0 .. P - 1 in order of part[p][i][j] (the split-k partial products).
__global__ __launch_bounds__(256) void sum_parts_kernel(int64_t M, int64_t Nc, int P, const double* __restrict__ part,
                                                        double* __restrict__ C, int64_t ldc) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= M * Nc) return;
  double acc = part[e];
  for (int p = 1; p < P; ++p) acc = acc + part[static_cast<int64_t>(p) * M * Nc + e];
  const int64_t i = e / Nc, j = e - i * Nc;
  C[i * ldc + j] = acc;
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

// out[0] = sum_{i < n} x[i] (the layer's QuantLoss from its per-row terms): one block, strided
// per-thread sums in index order, then the same fixed tree.
__global__ __launch_bounds__(256) void sum_f64_kernel(int64_t n, const double* __restrict__ x,
                                                      double* __restrict__ out) {
  __shared__ double red[256];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) acc = acc + x[i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w) red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0];
}

// ---- per-code sums ------------------------------------------------------------------------------
constexpr int kCsVec = 256;      // vectors staged per round
constexpr int kCsMaxOwn = 4;     // codes per thread (K <= 1024)
constexpr int64_t kCsMaxK = 256 * kCsMaxOwn;  // larger books are grouped by a radix pass (k_kmeans.hip)

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

// K <= 256, d <= 8: per-wave tables.  Every wave owns a private fp64 table of K x 8 sums in LDS and the
// batches of 64 vectors wave, wave + W, ... (W waves in the grid).  Within a batch the lanes that share
// a code find each other with eight ballots, and the lowest of them adds its peers' vectors (staged in
// LDS) in ascending lane order to that code's entry, so every entry is a fixed-order sum over the
// wave's batches; the block then folds its wave tables in wave order (layout [k * d + t][block]).
constexpr int kCwWaves = 6;   // waves per block: 6 tables of 21 KiB fit one CU's LDS
constexpr int kCwDepth = 2;   // batches in flight per wave

struct CwTable {
  double acc[256 * 8];
  int cnt[256];
  double stage[64][8];
};

__device__ __forceinline__ uint64_t code_peers(bool valid, int c) {
  uint64_t peers = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (c >> b) & 1;
    const uint64_t m = __ballot(bit);
    peers &= bit ? m : ~m;
  }
  return valid ? peers : 0ull;
}

__device__ __forceinline__ void cw_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// vector i of the set as 8 doubles (zero past d); a lane outside the set reads vector 0
__device__ __forceinline__ void cw_load(const double* X, int64_t vpr, int64_t ld, int d, int64_t i, bool ok,
                                        double (&v)[8]) {
  const int64_t j = ok ? i : 0;
  const int64_t r = j / vpr, g = j - r * vpr;
  const double* p = X + r * ld + g * d;
#pragma unroll
  for (int t = 0; t < 8; ++t) v[t] = t < d ? p[t] : 0.0;
}

__global__ __launch_bounds__(64 * kCwWaves) void code_sum_wave_partial(const double* __restrict__ X, int64_t vpr,
                                                                       int64_t ld, int d, int64_t n,
                                                                       const int32_t* __restrict__ codes, int K,
                                                                       int64_t nblocks, double* __restrict__ part,
                                                                       int* __restrict__ pcount) {
  __shared__ CwTable tab[kCwWaves];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  CwTable& T = tab[w];
  for (int e = lane; e < 256 * 8; e += 64) T.acc[e] = 0.0;
  for (int e = lane; e < 256; e += 64) T.cnt[e] = 0;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kCwWaves * 64;
  const int64_t w0 = (static_cast<int64_t>(blockIdx.x) * kCwWaves + w) * 64;
  double v[kCwDepth][8];
  int cq[kCwDepth];
#pragma unroll
  for (int s = 0; s < kCwDepth; ++s) {
    const int64_t i = w0 + stride * s + lane;
    const bool ok = i < n;
    cw_load(X, vpr, ld, d, i, ok, v[s]);
    cq[s] = codes[ok ? i : 0];
  }
  for (int64_t base = w0; base < n; base += stride * kCwDepth) {
#pragma unroll
    for (int s = 0; s < kCwDepth; ++s) {
      const int64_t bb = base + stride * s;
      if (bb < n) {  // uniform across the wave
        const int c = (bb + lane < n) ? cq[s] : -1;
        const bool valid = c >= 0 && c < K;
#pragma unroll
        for (int t = 0; t < 8; ++t) T.stage[lane][t] = v[s][t];
        cw_sync();
        const uint64_t peers = code_peers(valid, valid ? c : 0);
        if (valid && (__ffsll(static_cast<long long>(peers)) - 1) == lane) {
          double acc[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) acc[t] = T.acc[c * 8 + t];
          uint64_t m = peers;
          while (m) {
            const int sl = __ffsll(static_cast<long long>(m)) - 1;
            m &= m - 1;
#pragma unroll
            for (int t = 0; t < 8; ++t) acc[t] = acc[t] + T.stage[sl][t];
          }
#pragma unroll
          for (int t = 0; t < 8; ++t) T.acc[c * 8 + t] = acc[t];
          T.cnt[c] += __popcll(peers);
        }
        cw_sync();
      }
      const int64_t i = bb + stride * kCwDepth + lane;
      const bool ok = i < n;
      cw_load(X, vpr, ld, d, i, ok, v[s]);
      cq[s] = codes[ok ? i : 0];
    }
  }
  __syncthreads();
  for (int e = tid; e < K * d; e += 64 * kCwWaves) {
    const int k = e / d, t = e - k * d;
    double acc = 0.0;
#pragma unroll
    for (int ww = 0; ww < kCwWaves; ++ww) acc = acc + tab[ww].acc[k * 8 + t];
    part[static_cast<int64_t>(e) * nblocks + blockIdx.x] = acc;
    if (t == 0) {
      int cnt = 0;
#pragma unroll
      for (int ww = 0; ww < kCwWaves; ++ww) cnt += tab[ww].cnt[k];
      pcount[static_cast<int64_t>(k) * nblocks + blockIdx.x] = cnt;
    }
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

// The same step on an fp32 master of a bf16 codebook (set from the book at step 1), then the book as
// the master rounded to bf16, nearest-even (the master is finite here: rounding on its bits).
__global__ __launch_bounds__(256) void adam_bf16_kernel(int64_t n, uint16_t* __restrict__ C, float* __restrict__ master,
                                                        const double* __restrict__ grad, double scale,
                                                        double* __restrict__ m, double* __restrict__ v, double lr,
                                                        double b1, double b2, double bc1, double bc2, double eps,
                                                        int first) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n) return;
  const float x0 = first ? __uint_as_float(static_cast<uint32_t>(C[i]) << 16) : master[i];
  const double g = scale * grad[i];
  const double mi = b1 * m[i] + (1.0 - b1) * g;
  const double vi = b2 * v[i] + (1.0 - b2) * (g * g);
  m[i] = mi;
  v[i] = vi;
  const double mh = mi / bc1;
  const double vh = vi / bc2;
  const float x = static_cast<float>(static_cast<double>(x0) - lr * mh / (sqrt(vh) + eps));
  master[i] = x;
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7f800000u) != 0x7f800000u) u += 0x7fffu + ((u >> 16) & 1u);  // inf and NaN keep their bits
  C[i] = static_cast<uint16_t>(u >> 16);
}

// ---- width-1 code search, one block of column groups per launch ----------------------------------
constexpr int kRfRows = 8;      // rows per workgroup, one wave each
constexpr int kRfThreads = 64 * kRfRows;
constexpr int kRbCols = 64;     // columns per block (whole groups: 64 / d of them)

__device__ __forceinline__ double book_elem(const void* C, int type, int64_t i) {
  if (type == ET_F32) return static_cast<double>(static_cast<const float*>(C)[i]);
  return static_cast<double>(__uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(C)[i]) << 16));
}

// The groups of columns [c0, c0 + bw) in order, for rows blockIdx.x * 8 + wave.  With s = (R H)_g, the
// loss change of moving a group's code from c0 to c_k is
//   c_k^T Hgg c_k - 2 c_k . (s + Hgg c_cur) - (the same at c_cur),
// so the row takes the k minimising f(k) = a_k - 2 c_k . b with a_k = c_k^T Hgg c_k and
// b = s + Hgg c_cur (lowest k on ties).  The block's H and the rows' (R H) on the block's columns are
// held in LDS; a moved row subtracts delta = c_k - c_cur from its residual and delta^T H[g rows, c] from
// its (R H) on the block's later columns, and writes delta (zero if unmoved) to D, from which one
// product D H updates the columns after the block.  A code outside [0, K) leaves the group unchanged.
template <int DMAX>
__global__ __launch_bounds__(kRfThreads) void refine_block_kernel(int64_t M, int d, int64_t c0, int bw,
                                                                 double* __restrict__ R, int64_t ldr,
                                                                 const double* __restrict__ S, int64_t lds,
                                                                 const double* __restrict__ H, int64_t ldh,
                                                                 const void* __restrict__ Cb, int c_type, int K,
                                                                 int32_t* __restrict__ codes, int64_t ldq,
                                                                 double* __restrict__ D, int64_t ldd) {
  extern __shared__ double sm[];
  double* Cs = sm;                      // K * d
  double* Ak = Cs + K * d;              // K
  double* Hb = Ak + K;                  // kRbCols x kRbCols
  double* sS = Hb + kRbCols * kRbCols;  // kRfRows x kRbCols
  __shared__ double s_b[kRfRows][16];
  __shared__ double s_delta[kRfRows][16];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kRfRows;
  const int64_t r = r0 + w;
  for (int e = tid; e < K * d; e += kRfThreads) Cs[e] = book_elem(Cb, c_type, e);
  for (int e = tid; e < bw * bw; e += kRfThreads) {
    const int i = e / bw, j = e - i * bw;
    Hb[i * kRbCols + j] = H[(c0 + i) * ldh + c0 + j];
  }
  for (int e = tid; e < kRfRows * bw; e += kRfThreads) {
    const int rr = e / bw, c = e - rr * bw;
    sS[rr * kRbCols + c] = (r0 + rr < M) ? S[(r0 + rr) * lds + c0 + c] : 0.0;
  }
  __syncthreads();
  const int ng = bw / d;
  for (int gi = 0; gi < ng; ++gi) {
    const int cg = gi * d;
    for (int k = tid; k < K; k += kRfThreads) {
      double a = 0.0;
      for (int t = 0; t < d; ++t) {
        double h = 0.0;
        for (int u = 0; u < d; ++u) h = h + Hb[(cg + t) * kRbCols + cg + u] * Cs[k * d + u];
        a = a + Cs[k * d + t] * h;
      }
      Ak[k] = a;
    }
    const int64_t gq = c0 / d + gi;
    const int cur = r < M ? codes[r * ldq + gq] : -1;
    const bool active = cur >= 0 && cur < K;
    if (active && lane < d) {  // b = s + Hgg c_cur, one lane per element
      double h = 0.0;
      for (int u = 0; u < d; ++u) h = h + Hb[(cg + lane) * kRbCols + cg + u] * Cs[cur * d + u];
      s_b[w][lane] = sS[w * kRbCols + cg + lane] + h;
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
          R[r * ldr + c0 + cg + lane] = R[r * ldr + c0 + cg + lane] - delta;
          D[r * ldd + cg + lane] = delta;
        }
        if (lane == 0) codes[r * ldq + gq] = bk;
      }
    }
    if (!moved && r < M && lane < d) D[r * ldd + cg + lane] = 0.0;
    __syncthreads();
    if (moved) {
      for (int c = cg + d + lane; c < bw; c += 64) {
        double acc = 0.0;
        for (int t = 0; t < d; ++t) acc = acc + s_delta[w][t] * Hb[(cg + t) * kRbCols + c];
        sS[w * kRbCols + c] = sS[w * kRbCols + c] - acc;
      }
    }
    __syncthreads();
  }
}

// ---- the same search for books too large for one CU's LDS ------------------------------------------
// One group at a time over all rows: refine_scan_kernel finds, for 64 rows per workgroup and one slice
// of the codebook per grid row y, the k minimising f(k) = a_k - 2 c_k . b (the formulas and orders of
// refine_block_kernel, so the same values); refine_apply_kernel merges the slices (lowest k among equal
// values) and moves the rows' codes, updating R, D and the block's later columns of S = R H in memory.
constexpr int kRsRows = 64;      // rows per workgroup of the scan
constexpr int kRsTile = 256;     // codewords staged in LDS per round
constexpr int kRsMaxSlices = 8;  // codebook slices (grid y) at most

// Thread (rg, ks) = (tid % 16, tid / 16) scores rows 4 rg .. 4 rg + 3 against every sixteenth
// codeword of each staged round (so a codeword read from LDS serves four rows); the next round's
// codewords are loaded into registers while the current one is scored.
template <int DMAX>
__global__ __launch_bounds__(256) void refine_scan_kernel(int64_t M, int d, int64_t col, int64_t gq,
                                                          const double* __restrict__ S, int64_t lds,
                                                          const double* __restrict__ H, int64_t ldh,
                                                          const void* __restrict__ Cb, int c_type, int K, int slice,
                                                          const int32_t* __restrict__ codes, int64_t ldq,
                                                          double* __restrict__ bestF, int* __restrict__ bestK) {
  constexpr int kPer = kRsTile * DMAX / 256;  // staged elements per thread and round
  __shared__ double Hg[16 * 16];
  __shared__ double sb[kRsRows][16];
  __shared__ double Cs[kRsTile * DMAX];
  __shared__ double Ak[kRsTile];
  __shared__ double rf[16][kRsRows];
  __shared__ int rk[16][kRsRows];
  const int tid = threadIdx.x, rg = tid & 15, ks = tid >> 4;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kRsRows;
  const int k0 = static_cast<int>(blockIdx.y) * slice;
  const int k1 = k0 + slice < K ? k0 + slice : K;
  for (int e = tid; e < d * d; e += 256) Hg[e] = H[(col + e / d) * ldh + col + e % d];
  __syncthreads();
  // b = s + Hgg c_cur per row (a row with a code outside [0, K) takes no part)
  for (int e = tid; e < kRsRows * d; e += 256) {
    const int rr = e / d, t = e - rr * d;
    const int64_t r = r0 + rr;
    const int cur = r < M ? codes[r * ldq + gq] : -1;
    double v = 0.0;
    if (cur >= 0 && cur < K) {
      double h = 0.0;
      for (int u = 0; u < d; ++u) h = h + Hg[t * d + u] * book_elem(Cb, c_type, static_cast<int64_t>(cur) * d + u);
      v = S[r * lds + col + t] + h;
    }
    sb[rr][t] = v;
  }
  __syncthreads();
  double b[4][DMAX];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int t = 0; t < DMAX; ++t) b[q][t] = t < d ? sb[4 * rg + q][t] : 0.0;
  double best[4];
  int bk[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    best[q] = __builtin_inf();
    bk[q] = K;
  }
  // round kt's codewords as kPer elements per thread (element e = tid + 256 i of the round)
  double pf[kPer];
  auto fetch = [&](int kt) {
    const int64_t base = static_cast<int64_t>(kt) * d, lim = static_cast<int64_t>(k1) * d;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int64_t e = base + tid + 256 * i;
      pf[i] = e < lim ? book_elem(Cb, c_type, e) : 0.0;
    }
  };
  if (k0 < k1) fetch(k0);
  for (int kt = k0; kt < k1; kt += kRsTile) {
    const int tn = k1 - kt < kRsTile ? k1 - kt : kRsTile;
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (tid + 256 * i < tn * d) Cs[tid + 256 * i] = pf[i];
    __syncthreads();
    if (kt + kRsTile < k1) fetch(kt + kRsTile);  // in flight while this round is scored
    if (tid < tn) {  // a_k = c_k^T Hgg c_k
      double a = 0.0;
      for (int t = 0; t < d; ++t) {
        double h = 0.0;
        for (int u = 0; u < d; ++u) h = h + Hg[t * d + u] * Cs[tid * d + u];
        a = a + Cs[tid * d + t] * h;
      }
      Ak[tid] = a;
    }
    __syncthreads();
    for (int jj = ks; jj < tn; jj += 16) {
      double c[DMAX];
#pragma unroll
      for (int t = 0; t < DMAX; ++t) c[t] = t < d ? Cs[jj * d + t] : 0.0;
      const double a = Ak[jj];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        double dot = 0.0;
#pragma unroll
        for (int t = 0; t < DMAX; ++t)
          if (t < d) dot = dot + c[t] * b[q][t];
        const double f = a - 2.0 * dot;
        if (f < best[q]) {
          best[q] = f;
          bk[q] = kt + jj;
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    rf[ks][4 * rg + q] = best[q];
    rk[ks][4 * rg + q] = bk[q];
  }
  __syncthreads();
  if (tid < kRsRows && r0 + tid < M) {
    double f0 = rf[0][tid];
    int k = rk[0][tid];
    for (int q = 1; q < 16; ++q)
      if (rf[q][tid] < f0 || (rf[q][tid] == f0 && rk[q][tid] < k)) {
        f0 = rf[q][tid];
        k = rk[q][tid];
      }
    bestF[static_cast<int64_t>(blockIdx.y) * M + r0 + tid] = f0;
    bestK[static_cast<int64_t>(blockIdx.y) * M + r0 + tid] = k;
  }
}

template <int DMAX>
__global__ __launch_bounds__(256) void refine_apply_kernel(int64_t M, int d, int64_t c0, int cg, int bw, int64_t gq,
                                                           double* __restrict__ R, int64_t ldr, double* __restrict__ S,
                                                           int64_t lds, const double* __restrict__ H, int64_t ldh,
                                                           const void* __restrict__ Cb, int c_type, int K,
                                                           int32_t* __restrict__ codes, int64_t ldq,
                                                           double* __restrict__ D, int64_t ldd, int nslice,
                                                           const double* __restrict__ bestF,
                                                           const int* __restrict__ bestK) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (r >= M) return;
  const int cur = codes[r * ldq + gq];
  double best = __builtin_inf();
  int bk = K;
  for (int sl = 0; sl < nslice; ++sl) {
    const double f = bestF[static_cast<int64_t>(sl) * M + r];
    const int k = bestK[static_cast<int64_t>(sl) * M + r];
    if (f < best || (f == best && k < bk)) {
      best = f;
      bk = k;
    }
  }
  const bool moved = cur >= 0 && cur < K && bk < K && bk != cur;
  double delta[DMAX];
#pragma unroll
  for (int t = 0; t < DMAX; ++t) {
    delta[t] = 0.0;
    if (t < d && moved)
      delta[t] = book_elem(Cb, c_type, static_cast<int64_t>(bk) * d + t) -
                 book_elem(Cb, c_type, static_cast<int64_t>(cur) * d + t);
  }
#pragma unroll
  for (int t = 0; t < DMAX; ++t)
    if (t < d) D[r * ldd + cg + t] = delta[t];
  if (!moved) return;
  codes[r * ldq + gq] = bk;
#pragma unroll
  for (int t = 0; t < DMAX; ++t)
    if (t < d) R[r * ldr + c0 + cg + t] = R[r * ldr + c0 + cg + t] - delta[t];
  for (int c = cg + d; c < bw; ++c) {
    double acc = 0.0;
#pragma unroll
    for (int t = 0; t < DMAX; ++t)
      if (t < d) acc = acc + delta[t] * H[(c0 + cg + t) * ldh + c0 + c];
    S[r * lds + c0 + c] = S[r * lds + c0 + c] - acc;
  }
}

}  // namespace

// ---- launchers -----------------------------------------------------------------------------------
hipError_t launch_gemm_f64(int64_t M, int64_t Nc, int64_t Kd, const void* A, int a_type, bool trans_a, int64_t lda,
                           const void* B, int b_type, int64_t ldb, double* C, int64_t ldc, hipStream_t stream,
                           bool sub) {
  if (M <= 0 || Nc <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(cdiv(Nc, kGBN)), static_cast<unsigned>(cdiv(M, kGBM)));
#define CRVQ_GEMM(TA, TB, TR, SB)                                                                          \
  hipLaunchKernelGGL((gemm_f64_kernel<TA, TB, TR, SB>), grid, dim3(256), 0, stream, M, Nc, Kd,             \
                     static_cast<const TA*>(A), lda, static_cast<const TB*>(B), ldb, C, ldc, Kd, int64_t{0})
  if (a_type == ET_F32 && b_type == ET_F32 && !sub && trans_a && CRVQ_GEMM_MFMA) {
    // the Gram matrix X^T X of fp32 activations, widened exactly on load
    const dim3 gm(static_cast<unsigned>(cdiv(Nc, kMT)), static_cast<unsigned>(cdiv(M, kMT)));
    hipLaunchKernelGGL((gemm_f64_mfma_kernel<false, 4, float, float, true>), gm, dim3(256), 0, stream, M, Nc, Kd,
                       static_cast<const float*>(A), lda, static_cast<const float*>(B), ldb, C, ldc, Kd, int64_t{0});
  } else if (a_type == ET_F32 && b_type == ET_F32 && !sub) {
    if (trans_a) CRVQ_GEMM(float, float, true, false); else CRVQ_GEMM(float, float, false, false);
  } else if (a_type == ET_F64 && b_type == ET_F64 && !trans_a && CRVQ_GEMM_MFMA) {
    const dim3 gm(static_cast<unsigned>(cdiv(Nc, kMT)), static_cast<unsigned>(cdiv(M, kMT)));
    const dim3 gs(static_cast<unsigned>(cdiv(Nc, kMT / 2)), static_cast<unsigned>(cdiv(M, kMT / 2)));
    if (sub)
      hipLaunchKernelGGL((gemm_f64_mfma_kernel<true, 2>), gs, dim3(256), 0, stream, M, Nc, Kd,
                         static_cast<const double*>(A), lda, static_cast<const double*>(B), ldb, C, ldc, Kd, int64_t{0});
    else
      hipLaunchKernelGGL((gemm_f64_mfma_kernel<false, 4>), gm, dim3(256), 0, stream, M, Nc, Kd,
                         static_cast<const double*>(A), lda, static_cast<const double*>(B), ldb, C, ldc, Kd, int64_t{0});
  } else if (a_type == ET_F64 && b_type == ET_F64 && !(trans_a && sub)) {
    if (trans_a) CRVQ_GEMM(double, double, true, false);
    else if (sub) CRVQ_GEMM(double, double, false, true);
    else CRVQ_GEMM(double, double, false, false);
  } else {
    return hipErrorInvalidValue;
  }
#undef CRVQ_GEMM
  return hipGetLastError();
}

// C = A B (fp64, row-major, no transpose) split over k into P parts of at least 512 when the output
// grid alone is too small to fill the device; part products go to ws (P x M x Nc doubles) and are
// summed in part order, so the result does not depend on scheduling.
int64_t gemm_split_parts(int64_t M, int64_t Nc, int64_t Kd) {
  const int64_t tiles = CRVQ_GEMM_MFMA ? cdiv(Nc, kMT) * cdiv(M, kMT) : cdiv(Nc, kGBN) * cdiv(M, kGBM);
  int64_t P = tiles >= 256 ? 1 : cdiv(512, tiles);
  const int64_t maxp = Kd / 512 > 1 ? Kd / 512 : 1;
  return P < maxp ? P : maxp;
}

hipError_t launch_gemm_f64_split(int64_t M, int64_t Nc, int64_t Kd, const double* A, int64_t lda, const double* B,
                                 int64_t ldb, double* C, int64_t ldc, double* ws, hipStream_t stream) {
  if (M <= 0 || Nc <= 0) return hipSuccess;
  const int64_t P = gemm_split_parts(M, Nc, Kd);
  if (P <= 1) return launch_gemm_f64(M, Nc, Kd, A, ET_F64, false, lda, B, ET_F64, ldb, C, ldc, stream);
  const int64_t kchunk = cdiv(cdiv(Kd, P), kMK) * kMK;
  const int64_t parts = cdiv(Kd, kchunk);
  if (CRVQ_GEMM_MFMA) {
    const dim3 gm(static_cast<unsigned>(cdiv(Nc, kMT)), static_cast<unsigned>(cdiv(M, kMT)), static_cast<unsigned>(parts));
    hipLaunchKernelGGL((gemm_f64_mfma_kernel<false, 4>), gm, dim3(256), 0, stream, M, Nc, Kd, A, lda, B, ldb, ws, Nc,
                       kchunk, M * Nc);
  } else {
    const dim3 grid(static_cast<unsigned>(cdiv(Nc, kGBN)), static_cast<unsigned>(cdiv(M, kGBM)),
                    static_cast<unsigned>(parts));
    hipLaunchKernelGGL((gemm_f64_kernel<double, double, false, false>), grid, dim3(256), 0, stream, M, Nc, Kd, A, lda,
                       B, ldb, ws, Nc, kchunk, M * Nc);
  }
  hipLaunchKernelGGL(sum_parts_kernel, dim3(static_cast<unsigned>(cdiv(M * Nc, 256))), dim3(256), 0, stream, M, Nc,
                     static_cast<int>(parts), ws, C, ldc);
  return hipGetLastError();
}

hipError_t launch_row_dot(int64_t M, int64_t n, const double* A, int64_t lda, const double* B, int64_t ldb,
                          double* out, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(row_dot_kernel, dim3(static_cast<unsigned>(M)), dim3(256), 0, stream, n, A, lda, B, ldb, out);
  return hipGetLastError();
}

hipError_t launch_sum_f64(int64_t n, const double* x, double* out, hipStream_t stream) {
  hipLaunchKernelGGL(sum_f64_kernel, dim3(1), dim3(256), 0, stream, n, x, out);
  return hipGetLastError();
}

static int64_t code_sum_blocks(int64_t n) {
  const int64_t rounds = cdiv(n > 0 ? n : 1, kCsVec);
  return rounds < 1024 ? rounds : 1024;
}

// blocks of the per-wave scheme: at most one wave per batch of 64 vectors, 256 CUs' worth of waves
static int64_t code_sum_wave_blocks(int64_t n) {
  const int64_t batches = cdiv(n > 0 ? n : 1, 64);
  const int64_t waves = batches < 256 * kCwWaves ? batches : 256 * kCwWaves;
  return cdiv(waves, kCwWaves);
}

size_t code_sums_ws_bytes(int64_t n, int64_t K, int d) {
  if (K > kCsMaxK) return code_sums_large_ws_bytes(n, K);
  WsCursor c(nullptr);
  const int64_t nb = code_sum_blocks(n) > code_sum_wave_blocks(n) ? code_sum_blocks(n) : code_sum_wave_blocks(n);
  c.take<double>(static_cast<size_t>(nb * K * d));
  c.take<int>(static_cast<size_t>(nb * K));
  return c.used;
}

hipError_t launch_code_sums(const double* X, int64_t vpr, int64_t ld, int d, int64_t n, const int32_t* codes,
                            int64_t K, double* sums, int32_t* counts, void* ws, hipStream_t stream) {
  if (K > kCsMaxK) {
    RowSrc src;
    src.base = X;
    src.type = ET_F64;
    src.d = d;
    src.vpr = vpr;
    src.ld = ld;
    src.n = n;
    return launch_code_sums_large(src, codes, K, sums, counts, ws, stream);
  }
  if (K <= 256 && d <= 8 && n > 0) {
    WsCursor cw(ws);
    const int64_t nbw = code_sum_wave_blocks(n);
    const int64_t nbmax = code_sum_blocks(n) > nbw ? code_sum_blocks(n) : nbw;
    double* part = cw.take<double>(static_cast<size_t>(nbmax * K * d));
    int* pcount = cw.take<int>(static_cast<size_t>(nbmax * K));
    hipLaunchKernelGGL(code_sum_wave_partial, dim3(static_cast<unsigned>(nbw)), dim3(64 * kCwWaves), 0, stream, X, vpr,
                       ld, d, n, codes, static_cast<int>(K), nbw, part, pcount);
    hipLaunchKernelGGL(code_sum_final, dim3(static_cast<unsigned>(cdiv(K * d, 4))), dim3(256), 0, stream, part, pcount,
                       nbw, K, d, sums, counts);
    return hipGetLastError();
  }
  WsCursor cur(ws);
  int64_t nb = code_sum_blocks(n);
  const int64_t per_block = cdiv(cdiv(n > 0 ? n : 1, nb), kCsVec) * kCsVec;
  nb = cdiv(n > 0 ? n : 1, per_block);
  const int64_t nbmax = code_sum_blocks(n) > code_sum_wave_blocks(n) ? code_sum_blocks(n) : code_sum_wave_blocks(n);
  double* part = cur.take<double>(static_cast<size_t>(nbmax * K * d));
  int* pcount = cur.take<int>(static_cast<size_t>(nbmax * K));
  hipLaunchKernelGGL(code_sum_partial, dim3(static_cast<unsigned>(nb)), dim3(256), 0, stream, X, vpr, ld, d, n, codes,
                     static_cast<int>(K), per_block, nb, part, pcount);
  hipLaunchKernelGGL(code_sum_final, dim3(static_cast<unsigned>(cdiv(K * d, 4))), dim3(256), 0, stream, part, pcount,
                     nb, K, d, sums, counts);
  return hipGetLastError();
}

hipError_t launch_adam_bf16(int64_t n, uint16_t* C, float* master, const double* grad, double scale, double* m,
                            double* v, double lr, double b1, double b2, double bc1, double bc2, double eps, bool first,
                            hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(adam_bf16_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0, stream, n, C, master,
                     grad, scale, m, v, lr, b1, b2, bc1, bc2, eps, first ? 1 : 0);
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
  return static_cast<size_t>(K * d + K + kRbCols * kRbCols + kRfRows * kRbCols) * sizeof(double);
}

size_t refine_ws_bytes(int64_t M, int64_t n_cols, int64_t N) {
  return align256(static_cast<size_t>(M) * static_cast<size_t>(n_cols) * sizeof(double)) +
         align256(static_cast<size_t>(M) * kRbCols * sizeof(double)) +
         align256(static_cast<size_t>(gemm_split_parts(M, n_cols, N)) * static_cast<size_t>(M) *
                  static_cast<size_t>(n_cols) * sizeof(double)) +
         align256(static_cast<size_t>(kRsMaxSlices) * static_cast<size_t>(M) * sizeof(double)) +
         align256(static_cast<size_t>(kRsMaxSlices) * static_cast<size_t>(M) * sizeof(int));
}

// The codebook fits the block kernel's LDS (with H's block and the rows' S).
bool refine_book_in_lds(int64_t K, int d) { return K * d <= 8192 && refine_lds_bytes(K, d) + 4096 <= 160 * 1024; }

hipError_t launch_refine_book(int64_t M, int64_t N, int d, int64_t n_cols, double* R, int64_t ldr, const double* H,
                              int64_t ldh, const void* Cb, int c_type, int64_t K, int32_t* codes, int64_t ldq,
                              void* ws, hipStream_t stream) {
  if (M <= 0 || n_cols <= 0) return hipSuccess;
  WsCursor cur(ws);
  double* S = cur.take<double>(static_cast<size_t>(M) * static_cast<size_t>(n_cols));
  double* D = cur.take<double>(static_cast<size_t>(M) * kRbCols);
  double* parts = cur.take<double>(static_cast<size_t>(gemm_split_parts(M, n_cols, N)) * static_cast<size_t>(M) *
                                   static_cast<size_t>(n_cols));
  double* bestF = cur.take<double>(static_cast<size_t>(kRsMaxSlices) * static_cast<size_t>(M));
  int* bestK = cur.take<int>(static_cast<size_t>(kRsMaxSlices) * static_cast<size_t>(M));
  // S = R H[:, 0:n_cols]
  hipError_t e = launch_gemm_f64_split(M, n_cols, N, R, ldr, H, ldh, S, n_cols, parts, stream);
  if (e != hipSuccess) return e;
  const size_t lds = refine_lds_bytes(K, d);
  const dim3 grid(static_cast<unsigned>(cdiv(M, kRfRows)));
  const int64_t bw_max = (kRbCols / d) * d;
  const bool in_lds = refine_book_in_lds(K, d);
  // large books: enough codebook slices to give the scan about 512 workgroups
  const int64_t row_tiles = cdiv(M, kRsRows);
  int64_t nslice = cdiv(512, row_tiles);
  nslice = nslice < kRsMaxSlices ? nslice : kRsMaxSlices;
  nslice = nslice < cdiv(K, kRsTile) ? nslice : cdiv(K, kRsTile);
  const int slice = static_cast<int>(cdiv(cdiv(K, nslice), kRsTile) * kRsTile);
  nslice = cdiv(K, slice);
  for (int64_t c0 = 0; c0 < n_cols; c0 += bw_max) {
    const int bw = static_cast<int>(n_cols - c0 < bw_max ? n_cols - c0 : bw_max);
    if (!in_lds) {
      for (int cg = 0; cg < bw; cg += d) {
        const int64_t gq = c0 / d + cg / d;
        const dim3 gs(static_cast<unsigned>(row_tiles), static_cast<unsigned>(nslice));
        const unsigned ga = static_cast<unsigned>(cdiv(M, 256));
        if (d <= 8) {
          hipLaunchKernelGGL(refine_scan_kernel<8>, gs, dim3(256), 0, stream, M, d, c0 + cg, gq, S, n_cols, H, ldh, Cb,
                             c_type, static_cast<int>(K), slice, codes, ldq, bestF, bestK);
          hipLaunchKernelGGL(refine_apply_kernel<8>, dim3(ga), dim3(256), 0, stream, M, d, c0, cg, bw, gq, R, ldr, S,
                             n_cols, H, ldh, Cb, c_type, static_cast<int>(K), codes, ldq, D, bw_max,
                             static_cast<int>(nslice), bestF, bestK);
        } else {
          hipLaunchKernelGGL(refine_scan_kernel<16>, gs, dim3(256), 0, stream, M, d, c0 + cg, gq, S, n_cols, H, ldh,
                             Cb, c_type, static_cast<int>(K), slice, codes, ldq, bestF, bestK);
          hipLaunchKernelGGL(refine_apply_kernel<16>, dim3(ga), dim3(256), 0, stream, M, d, c0, cg, bw, gq, R, ldr, S,
                             n_cols, H, ldh, Cb, c_type, static_cast<int>(K), codes, ldq, D, bw_max,
                             static_cast<int>(nslice), bestF, bestK);
        }
      }
    } else if (d <= 8)
      hipLaunchKernelGGL(refine_block_kernel<8>, grid, dim3(kRfThreads), lds, stream, M, d, c0, bw, R, ldr, S, n_cols,
                         H, ldh, Cb, c_type, static_cast<int>(K), codes, ldq, D, bw_max);
    else
      hipLaunchKernelGGL(refine_block_kernel<16>, grid, dim3(kRfThreads), lds, stream, M, d, c0, bw, R, ldr, S, n_cols,
                         H, ldh, Cb, c_type, static_cast<int>(K), codes, ldq, D, bw_max);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // the block's code changes reach the later columns: S[:, c0 + bw :] -= D H[c0 .. c0 + bw, c0 + bw :]
    if (c0 + bw < n_cols) {
      e = launch_gemm_f64(M, n_cols - c0 - bw, bw, D, ET_F64, false, bw_max, H + c0 * ldh + c0 + bw, ET_F64, ldh,
                          S + c0 + bw, n_cols, stream, true);
      if (e != hipSuccess) return e;
    }
  }
  return hipGetLastError();
}

}  // namespace crvq
