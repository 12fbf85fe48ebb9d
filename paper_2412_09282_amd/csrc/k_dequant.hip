// Additive reconstruction of CRVQ codes (Sec. 4.3 of the paper): a vector of a critical group is
// the sum of its basic and extended codewords, any other vector its basic codeword.  The same
// kernel produces the residual E = minuend - reconstruction (Alg. 1 ComputeError / Update) and the
// reverse reordering back to the original channel order (Sec. 4.3, Fig. 3 right).
//
// One block per row.  Every element is summed in fp64 in book order and rounded once.  With a
// permutation the rounded row is staged in LDS and written out in original channel order through
// the inverse permutation, so both the codebook reads and the output writes stay coalesced.
#include "crvq_internal.h"

namespace crvq {
namespace {

__device__ __forceinline__ double elem(const void* p, int type, int64_t i) {
  if (type == ET_F32) return static_cast<double>(static_cast<const float*>(p)[i]);
  return static_cast<double>(__uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(p)[i]) << 16));
}

__device__ __forceinline__ uint16_t bf16_from_double(double x) {
  const double ax = fabs(x);
  if (!(ax >= 0x1p-126)) {
    if (x != x) return 0x7fc0;
    const double r = rint(x * 0x1p133) * 0x1p-133;
    return static_cast<uint16_t>(__float_as_uint(static_cast<float>(r)) >> 16);
  }
  uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
  const uint64_t lsb = (u >> 45) & 1;
  u += (1ull << 44) - 1 + lsb;
  u &= ~((1ull << 45) - 1);
  const float f = static_cast<float>(__longlong_as_double(static_cast<long long>(u)));
  return static_cast<uint16_t>(__float_as_uint(f) >> 16);
}

// fp64 reconstruction of element c of row r (NaN if a code is out of range).
__device__ __forceinline__ double recon(const DequantBooks& b, int64_t r, int64_t c, int d, int64_t n_crit_vec) {
  const int64_t g = c / d;
  const int t = static_cast<int>(c - g * d);
  const int32_t q0 = b.q[0][r * b.ldq_base + g];
  if (q0 < 0 || q0 >= b.K[0]) return __builtin_nan("");
  double v = elem(b.C[0], b.type[0], static_cast<int64_t>(q0) * d + t);
  if (g < n_crit_vec) {
    for (int e = 1; e < b.n; ++e) {
      const int32_t q = b.q[e][r * b.ldq_ext + g];
      if (q < 0 || q >= b.K[e]) return __builtin_nan("");
      v = v + elem(b.C[e], b.type[e], static_cast<int64_t>(q) * d + t);
    }
  }
  return v;
}

__global__ __launch_bounds__(256) void dequant_rows(int64_t n_cols, int d, int64_t n_crit_vec, DequantBooks b,
                                                    const void* __restrict__ minuend, int min_type, int64_t ld_min,
                                                    void* __restrict__ out, int out_type, int64_t ld_out) {
  const int64_t r = blockIdx.x;
  for (int64_t c = threadIdx.x; c < n_cols; c += 256) {
    double v = recon(b, r, c, d, n_crit_vec);
    if (minuend) v = elem(minuend, min_type, r * ld_min + c) - v;
    if (out_type == ET_F32)
      static_cast<float*>(out)[r * ld_out + c] = static_cast<float>(v);
    else
      static_cast<uint16_t*>(out)[r * ld_out + c] = bf16_from_double(v);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void dequant_rows_perm(int64_t n_cols, int d, int64_t n_crit_vec, DequantBooks b,
                                                         const int32_t* __restrict__ inv, T* __restrict__ out,
                                                         int64_t ld_out) {
  extern __shared__ unsigned char smem[];
  T* row = reinterpret_cast<T*>(smem);
  const int64_t r = blockIdx.x;
  for (int64_t c = threadIdx.x; c < n_cols; c += 256) {
    const double v = recon(b, r, c, d, n_crit_vec);
    if constexpr (sizeof(T) == 4)
      row[c] = __float_as_uint(static_cast<float>(v));
    else
      row[c] = bf16_from_double(v);
  }
  __syncthreads();
  for (int64_t j = threadIdx.x; j < n_cols; j += 256) {
    const int32_t s = inv[j];
    if (s >= 0 && s < n_cols) out[r * ld_out + j] = row[s];
  }
}

// Rows too long for LDS: scatter straight to the permuted column.
__global__ __launch_bounds__(256) void dequant_perm_direct(int64_t M, int64_t n_cols, int d, int64_t n_crit_vec,
                                                           DequantBooks b, const int32_t* __restrict__ inv,
                                                           void* __restrict__ out, int out_type, int64_t ld_out) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= M * n_cols) return;
  const int64_t r = e / n_cols;
  const int64_t j = e - r * n_cols;
  const int32_t s = inv[j];
  if (s < 0 || s >= n_cols) return;
  const double v = recon(b, r, s, d, n_crit_vec);
  if (out_type == ET_F32)
    static_cast<float*>(out)[r * ld_out + j] = static_cast<float>(v);
  else
    static_cast<uint16_t*>(out)[r * ld_out + j] = bf16_from_double(v);
}

}  // namespace

hipError_t launch_dequant(int64_t M, int64_t n_cols, int d, int64_t n_crit, const DequantBooks& books,
                          const int32_t* inv_perm, const void* minuend, int min_type, int64_t ld_min, void* out,
                          int out_type, int64_t ld_out, hipStream_t stream) {
  if (M <= 0 || n_cols <= 0) return hipSuccess;
  const int64_t ncv = n_crit / d;
  if (!inv_perm) {
    hipLaunchKernelGGL(dequant_rows, dim3(static_cast<unsigned>(M)), dim3(256), 0, stream, n_cols, d, ncv, books, minuend,
                       min_type, ld_min, out, out_type, ld_out);
  } else {
    const int esize = out_type == ET_F32 ? 4 : 2;
    const size_t lds = static_cast<size_t>(n_cols) * esize;
    if (lds <= 64 * 1024) {
      if (esize == 4)
        hipLaunchKernelGGL(dequant_rows_perm<uint32_t>, dim3(static_cast<unsigned>(M)), dim3(256), lds, stream, n_cols, d,
                           ncv, books, inv_perm, static_cast<uint32_t*>(out), ld_out);
      else
        hipLaunchKernelGGL(dequant_rows_perm<uint16_t>, dim3(static_cast<unsigned>(M)), dim3(256), lds, stream, n_cols, d,
                           ncv, books, inv_perm, static_cast<uint16_t*>(out), ld_out);
    } else {
      hipLaunchKernelGGL(dequant_perm_direct, dim3(static_cast<unsigned>(cdiv(M * n_cols, 256))), dim3(256), 0, stream, M,
                         n_cols, d, ncv, books, inv_perm, out, out_type, ld_out);
    }
  }
  return hipGetLastError();
}

}  // namespace crvq
