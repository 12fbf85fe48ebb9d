// Additive reconstruction of CRVQ codes (Sec. 4.3 of the paper): a vector of a critical group is
// the sum of its basic and extended codewords, any other vector its basic codeword.  The same
// kernels produce the residual E = minuend - reconstruction (Alg. 1 ComputeError / Update) and the
// reverse reordering back to the original channel order (Sec. 4.3, Fig. 3 right).
//
// One thread per d-vector: its codes are read once, each codeword as one contiguous piece, every
// element summed in fp64 in book order and rounded once.  With a permutation the block rebuilds a
// whole row in LDS and writes it out in original channel order through the inverse permutation,
// 16 bytes per thread and store, so codebook reads and output writes stay coalesced.
#include "crvq_internal.h"

namespace crvq {
namespace {

constexpr int kMaxD = 16;

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

// Adds codeword q of book b (d elements) to v in fp64; fp32 books with d % 4 == 0 are read as float4.
__device__ __forceinline__ void add_codeword(const void* C, int type, int64_t q, int d, double (&v)[kMaxD]) {
  if (type == ET_F32 && (d & 3) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0) {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(C) + q * d);
#pragma unroll
    for (int t4 = 0; t4 < kMaxD / 4; ++t4) {
      if (4 * t4 < d) {
        const float4 w = p[t4];
        v[4 * t4] = v[4 * t4] + static_cast<double>(w.x);
        v[4 * t4 + 1] = v[4 * t4 + 1] + static_cast<double>(w.y);
        v[4 * t4 + 2] = v[4 * t4 + 2] + static_cast<double>(w.z);
        v[4 * t4 + 3] = v[4 * t4 + 3] + static_cast<double>(w.w);
      }
    }
  } else {
#pragma unroll
    for (int t = 0; t < kMaxD; ++t)
      if (t < d) v[t] = v[t] + elem(C, type, q * d + t);
  }
}

// fp64 reconstruction of vector g of row r; returns false (NaN row) if a code is out of range.
__device__ __forceinline__ bool recon_vec(const DequantBooks& b, int64_t r, int64_t g, int d, int64_t n_crit_vec,
                                          double (&v)[kMaxD]) {
#pragma unroll
  for (int t = 0; t < kMaxD; ++t) v[t] = 0.0;
  const int32_t q0 = b.q[0][r * b.ldq_base + g];
  if (q0 < 0 || q0 >= b.K[0]) return false;
  add_codeword(b.C[0], b.type[0], q0, d, v);
  if (g < n_crit_vec) {
    for (int e = 1; e < b.n; ++e) {
      const int32_t q = b.q[e][r * b.ldq_ext + g];
      if (q < 0 || q >= b.K[e]) return false;
      add_codeword(b.C[e], b.type[e], q, d, v);
    }
  }
  return true;
}

__global__ __launch_bounds__(256) void dequant_rows(int64_t M, int64_t n_cols, int d, int64_t n_crit_vec,
                                                    DequantBooks b, const void* __restrict__ minuend, int min_type,
                                                    int64_t ld_min, void* __restrict__ out, int out_type,
                                                    int64_t ld_out) {
  const int64_t vpr = n_cols / d;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= M * vpr) return;
  const int64_t r = e / vpr;
  const int64_t g = e - r * vpr;
  double v[kMaxD];
  const bool ok = recon_vec(b, r, g, d, n_crit_vec, v);
  const int64_t c0 = g * d;
#pragma unroll
  for (int t = 0; t < kMaxD; ++t) {
    if (t < d) {
      double x = ok ? v[t] : __builtin_nan("");
      if (minuend) x = elem(minuend, min_type, r * ld_min + c0 + t) - x;
      if (out_type == ET_F32)
        static_cast<float*>(out)[r * ld_out + c0 + t] = static_cast<float>(x);
      else
        static_cast<uint16_t*>(out)[r * ld_out + c0 + t] = bf16_from_double(x);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void dequant_rows_perm(int64_t n_cols, int d, int64_t n_crit_vec, DequantBooks b,
                                                         const int32_t* __restrict__ inv, T* __restrict__ out,
                                                         int64_t ld_out, int vec_out) {
  extern __shared__ unsigned char smem[];
  T* row = reinterpret_cast<T*>(smem);
  const int64_t r = blockIdx.x;
  const int64_t vpr = n_cols / d;
  for (int64_t g = threadIdx.x; g < vpr; g += 256) {
    double v[kMaxD];
    const bool ok = recon_vec(b, r, g, d, n_crit_vec, v);
#pragma unroll
    for (int t = 0; t < kMaxD; ++t) {
      if (t < d) {
        const double x = ok ? v[t] : __builtin_nan("");
        if constexpr (sizeof(T) == 4)
          row[g * d + t] = __float_as_uint(static_cast<float>(x));
        else
          row[g * d + t] = bf16_from_double(x);
      }
    }
  }
  __syncthreads();
  T* ro = out + r * ld_out;
  if (vec_out) {  // 16-byte segments of the output row
    constexpr int V = 16 / sizeof(T);
    for (int64_t c = threadIdx.x; c < n_cols / V; c += 256) {
      T seg[V];
#pragma unroll
      for (int q = 0; q < V; q += 4) {
        const int4 s4 = reinterpret_cast<const int4*>(inv)[(c * V + q) / 4];
        const int32_t s[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) seg[q + u] = (s[u] >= 0 && s[u] < n_cols) ? row[s[u]] : T(0);
      }
      reinterpret_cast<uint4*>(ro)[c] = *reinterpret_cast<const uint4*>(seg);
    }
  } else {
    for (int64_t j = threadIdx.x; j < n_cols; j += 256) {
      const int32_t s = inv[j];
      if (s >= 0 && s < n_cols) ro[j] = row[s];
    }
  }
}

// Rows too long for LDS: one thread per d-vector, scattered to the permuted columns.
__global__ __launch_bounds__(256) void dequant_perm_direct(int64_t M, int64_t n_cols, int d, int64_t n_crit_vec,
                                                           DequantBooks b, const int32_t* __restrict__ perm,
                                                           void* __restrict__ out, int out_type, int64_t ld_out) {
  const int64_t vpr = n_cols / d;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= M * vpr) return;
  const int64_t r = e / vpr;
  const int64_t g = e - r * vpr;
  double v[kMaxD];
  const bool ok = recon_vec(b, r, g, d, n_crit_vec, v);
#pragma unroll
  for (int t = 0; t < kMaxD; ++t) {
    if (t < d) {
      const int32_t j = perm[g * d + t];
      if (j < 0 || j >= n_cols) continue;
      const double x = ok ? v[t] : __builtin_nan("");
      if (out_type == ET_F32)
        static_cast<float*>(out)[r * ld_out + j] = static_cast<float>(x);
      else
        static_cast<uint16_t*>(out)[r * ld_out + j] = bf16_from_double(x);
    }
  }
}

}  // namespace

hipError_t launch_dequant(int64_t M, int64_t n_cols, int d, int64_t n_crit, const DequantBooks& books,
                          const int32_t* inv_perm, const int32_t* perm, const void* minuend, int min_type,
                          int64_t ld_min, void* out, int out_type, int64_t ld_out, hipStream_t stream) {
  if (M <= 0 || n_cols <= 0) return hipSuccess;
  const int64_t ncv = n_crit / d;
  const int64_t nvec = M * (n_cols / d);
  if (!inv_perm) {
    hipLaunchKernelGGL(dequant_rows, dim3(static_cast<unsigned>(cdiv(nvec, 256))), dim3(256), 0, stream, M, n_cols, d, ncv,
                       books, minuend, min_type, ld_min, out, out_type, ld_out);
  } else {
    const int esize = out_type == ET_F32 ? 4 : 2;
    const size_t lds = static_cast<size_t>(n_cols) * esize;
    const int V = 16 / esize;
    const int vec_out = (n_cols % V == 0) && ((ld_out * esize) % 16 == 0) &&
                        (reinterpret_cast<uintptr_t>(out) % 16 == 0) && (reinterpret_cast<uintptr_t>(inv_perm) % 16 == 0);
    if (lds <= 64 * 1024) {
      if (esize == 4)
        hipLaunchKernelGGL(dequant_rows_perm<uint32_t>, dim3(static_cast<unsigned>(M)), dim3(256), lds, stream, n_cols, d,
                           ncv, books, inv_perm, static_cast<uint32_t*>(out), ld_out, vec_out);
      else
        hipLaunchKernelGGL(dequant_rows_perm<uint16_t>, dim3(static_cast<unsigned>(M)), dim3(256), lds, stream, n_cols, d,
                           ncv, books, inv_perm, static_cast<uint16_t*>(out), ld_out, vec_out);
    } else {
      hipLaunchKernelGGL(dequant_perm_direct, dim3(static_cast<unsigned>(cdiv(nvec, 256))), dim3(256), 0, stream, M,
                         n_cols, d, ncv, books, perm, out, out_type, ld_out);
    }
  }
  return hipGetLastError();
}

}  // namespace crvq
