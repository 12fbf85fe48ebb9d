// Additive reconstruction of CRVQ codes (Sec. 4.3 of the paper): a vector of a critical group is
// the sum of its basic and extended codewords, any other vector its basic codeword.  The same
// kernels produce the residual E = minuend - reconstruction (Alg. 1 ComputeError / Update) and the
// reverse reordering back to the original channel order (Sec. 4.3, Fig. 3 right).
//
// Every element is summed in fp64 in book order and rounded once.  d = 8 (the common case): two
// lanes per vector, each gathering and writing one 16-byte half, codes and outputs streamed with
// nontemporal accesses; with a permutation, persistent blocks rebuild one row at a time in LDS and
// write it out in original channel order through the inverse permutation (kept in LDS), 16 bytes
// per store.  Other d, and layouts with several basic books: one thread per vector with the same
// arithmetic.
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
  for (int e = 0; e < b.n_full; ++e) {
    const int32_t q = b.q[e][r * b.ldq_base + g];
    if (q < 0 || q >= b.K[e]) return false;
    add_codeword(b.C[e], b.type[e], q, d, v);
  }
  if (g < n_crit_vec) {
    for (int e = b.n_full; e < b.n; ++e) {
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
      else if (out_type == ET_F64)
        static_cast<double*>(out)[r * ld_out + c0 + t] = x;
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

// ---- d = 8 with 16-byte aligned books and rows: the same arithmetic, two lanes per vector.  Lane
// half h of a pair reads and writes dimensions 4h .. 4h + 3, so both halves of a codeword gather
// come from one cache line and every store of a wave is one contiguous piece.  All code and
// codeword loads of a thread's vectors are issued before any is used.

// Half h (4 elements) of codeword q as floats: one float4 (fp32) or one 8-byte load (bf16).
__device__ __forceinline__ void load_cw4(const void* C, int type, int64_t q, int h, float (&c)[4]) {
  if (type == ET_F32) {
    const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(C) + q * 8 + 4 * h);
    c[0] = a.x; c[1] = a.y; c[2] = a.z; c[3] = a.w;
  } else {
    const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(C) + q * 8 + 4 * h);
    c[0] = __uint_as_float(w.x << 16);
    c[1] = __uint_as_float(w.x & 0xffff0000u);
    c[2] = __uint_as_float(w.y << 16);
    c[3] = __uint_as_float(w.y & 0xffff0000u);
  }
}

// fp64 reconstruction of half h of vector g of row r from its (already loaded) basic codeword
// half c0: the extended books of a critical vector are added in book order.  Returns false (NaN
// vector) on a code out of range.
__device__ __forceinline__ bool recon4(const DequantBooks& b, int64_t r, int64_t g, int h, int64_t ncv, bool ok0,
                                       const float (&c0)[4], double (&v)[4]) {
#pragma unroll
  for (int t = 0; t < 4; ++t) v[t] = 0.0 + static_cast<double>(c0[t]);
  bool ok = ok0;
  if (g < ncv) {
    for (int e = 1; e < b.n; ++e) {
      const int32_t q = b.q[e][r * b.ldq_ext + g];
      const bool in = q >= 0 && q < b.K[e];
      ok = ok && in;
      float c[4];
      load_cw4(b.C[e], b.type[e], in ? q : 0, h, c);
#pragma unroll
      for (int t = 0; t < 4; ++t) v[t] = v[t] + static_cast<double>(c[t]);
    }
  }
  return ok;
}

// 4 output elements from fp64 values (fp32: 16 bytes, bf16: 8 bytes).  STREAM: a global output
// written once (nontemporal); otherwise plain stores (LDS).
template <typename T, bool STREAM>
__device__ __forceinline__ void store4(T* p, const double (&x)[4]) {
  if constexpr (sizeof(T) == 4) {
    uint4 a;
    a.x = __float_as_uint(static_cast<float>(x[0]));
    a.y = __float_as_uint(static_cast<float>(x[1]));
    a.z = __float_as_uint(static_cast<float>(x[2]));
    a.w = __float_as_uint(static_cast<float>(x[3]));
    if (STREAM)
      st_stream(p, a);
    else
      *reinterpret_cast<uint4*>(p) = a;
  } else {
    uint2 w;
    w.x = static_cast<uint32_t>(bf16_from_double(x[0])) | (static_cast<uint32_t>(bf16_from_double(x[1])) << 16);
    w.y = static_cast<uint32_t>(bf16_from_double(x[2])) | (static_cast<uint32_t>(bf16_from_double(x[3])) << 16);
    *reinterpret_cast<uint2*>(p) = w;
  }
}

// Two lanes per vector, reconstruction or residual (minuend - reconstruction), no permutation.
template <typename T, typename TM>
__global__ __launch_bounds__(256) void dequant_rows8(int64_t M, int64_t vpr, int64_t ncv, DequantBooks b,
                                                     const TM* __restrict__ minuend, int64_t ld_min,
                                                     T* __restrict__ out, int64_t ld_out) {
  const int64_t e2 = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e2 >= 2 * M * vpr) return;
  const int h = static_cast<int>(e2 & 1);
  const int64_t e = e2 >> 1;
  const int64_t r = e / vpr;
  const int64_t g = e - r * vpr;
  const int32_t q0 = ld_stream_i32(b.q[0] + r * b.ldq_base + g);
  float m[4];
  if (minuend) {
    if constexpr (sizeof(TM) == 4) {
      const uint4 a = ld_stream(minuend + r * ld_min + g * 8 + 4 * h);
      m[0] = __uint_as_float(a.x); m[1] = __uint_as_float(a.y); m[2] = __uint_as_float(a.z); m[3] = __uint_as_float(a.w);
    } else {
      const uint2 w = ld_stream8(minuend + r * ld_min + g * 8 + 4 * h);
      m[0] = __uint_as_float(w.x << 16);
      m[1] = __uint_as_float(w.x & 0xffff0000u);
      m[2] = __uint_as_float(w.y << 16);
      m[3] = __uint_as_float(w.y & 0xffff0000u);
    }
  }
  const bool in = q0 >= 0 && q0 < b.K[0];
  float c0[4];
  load_cw4(b.C[0], b.type[0], in ? q0 : 0, h, c0);
  double v[4];
  const bool ok = recon4(b, r, g, h, ncv, in, c0, v);
  double x[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    x[t] = ok ? v[t] : __builtin_nan("");
    if (minuend) x[t] = static_cast<double>(m[t]) - x[t];
  }
  store4<T, true>(out + r * ld_out + g * 8 + 4 * h, x);
}

// Reconstruction in original channel order.  Persistent blocks of 512 threads keep the inverse
// permutation in LDS (16-bit column indices, read from memory once per block) and walk rows
// r = block, block + grid, ...: each row is rebuilt in LDS (kUP vectors per lane pair and round, so a
// row of up to 8192 columns takes one round), then written through the inverse permutation in
// 16-byte segments.  This form takes any books; the extended codes of a critical vector are read
// where it is rebuilt.
constexpr int kPermThreads = 512;
constexpr int kUP = 4;  // vectors per lane pair and round in the permuted-row kernels
constexpr int kPE = 2;  // extended books handled by the specialised kernel

template <typename T>
__global__ __launch_bounds__(kPermThreads) void dequant_rows_perm8(int64_t M, int64_t n_cols, int64_t ncv,
                                                                   DequantBooks b, const int32_t* __restrict__ inv,
                                                                   T* __restrict__ out, int64_t ld_out) {
  extern __shared__ unsigned char smem[];
  T* row = reinterpret_cast<T*>(smem);
  uint16_t* src = reinterpret_cast<uint16_t*>(smem + ((n_cols * sizeof(T) + 15) & ~static_cast<int64_t>(15)));
  for (int64_t j = threadIdx.x; j < n_cols; j += kPermThreads) {
    const int32_t sj = inv[j];
    src[j] = (sj >= 0 && sj < n_cols) ? static_cast<uint16_t>(sj) : static_cast<uint16_t>(0xffff);  // 0xffff: zero
  }
  const int64_t vpr = n_cols / 8;
  const int h = threadIdx.x & 1;
  const int pair = threadIdx.x >> 1;
  constexpr int kPairs = kPermThreads / 2;
  constexpr int V = 16 / sizeof(T);
  for (int64_t r = blockIdx.x; r < M; r += gridDim.x) {
    for (int64_t g0 = pair; g0 < vpr; g0 += kPairs * kUP) {
      int32_t q[kUP];
      bool live[kUP], in[kUP];
#pragma unroll
      for (int u = 0; u < kUP; ++u) {
        const int64_t g = g0 + kPairs * u;
        live[u] = g < vpr;
        q[u] = live[u] ? ld_stream_i32(b.q[0] + r * b.ldq_base + g) : 0;
      }
      float c[kUP][4];
#pragma unroll
      for (int u = 0; u < kUP; ++u) {
        in[u] = q[u] >= 0 && q[u] < b.K[0];
        load_cw4(b.C[0], b.type[0], (live[u] && in[u]) ? q[u] : 0, h, c[u]);
      }
#pragma unroll
      for (int u = 0; u < kUP; ++u) {
        const int64_t g = g0 + kPairs * u;
        if (!live[u]) continue;
        double v[4];
        const bool ok = recon4(b, r, g, h, ncv, in[u], c[u], v);
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = ok ? v[t] : __builtin_nan("");
        store4<T, false>(row + g * 8 + 4 * h, v);
      }
    }
    __syncthreads();  // the row (and, first time round, the permutation) is in LDS
    T* ro = out + r * ld_out;
    for (int64_t c = threadIdx.x; c < n_cols / V; c += kPermThreads) {
      T seg[V];
#pragma unroll
      for (int u = 0; u < V; ++u) {
        const uint32_t sj = src[c * V + u];
        seg[u] = (sj < static_cast<uint32_t>(n_cols)) ? row[sj] : T(0);
      }
      st_stream(reinterpret_cast<uint4*>(ro) + c, *reinterpret_cast<const uint4*>(seg));
    }
    __syncthreads();  // the row buffer is rewritten by the next row
  }
}

// The same kernel specialised for the common case, with every load of a round straight-line code
// (no branch between a load and its use, so all of a round's gathers are in flight together; no
// prefetch across rows either: waiting for codes loaded before a row's stores would also wait for
// those stores):
// basic book element type TB, exactly NE extended books (fp32), critical groups of a row within
// the first 256 vectors (only a lane pair's first vector of a round can be critical).  Loads of
// absent entries read a valid address (code 0, vector 0) and their values are discarded.
template <typename TB>
__device__ __forceinline__ void load_cw4t(const TB* C, int32_t q, int h, float (&c)[4]) {
  if constexpr (sizeof(TB) == 4) {
    const float4 a = *reinterpret_cast<const float4*>(C + static_cast<int64_t>(q) * 8 + 4 * h);
    c[0] = a.x; c[1] = a.y; c[2] = a.z; c[3] = a.w;
  } else {
    const uint2 w = *reinterpret_cast<const uint2*>(C + static_cast<int64_t>(q) * 8 + 4 * h);
    c[0] = __uint_as_float(w.x << 16);
    c[1] = __uint_as_float(w.x & 0xffff0000u);
    c[2] = __uint_as_float(w.y << 16);
    c[3] = __uint_as_float(w.y & 0xffff0000u);
  }
}

// 4 output elements from fp32 values: a vector with one codeword is that codeword, so its fp64 sum
// rounds back to the same fp32 value (bf16: the same nearest-even rounding of the fp32 value).
__device__ __forceinline__ uint16_t bf16_from_float(float x) {
  const uint32_t u = __float_as_uint(x);
  if (x != x) return 0x7fc0;
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}
template <typename T>
__device__ __forceinline__ void store4f(T* p, const float (&x)[4]) {
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<uint4*>(p) =
        make_uint4(__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]), __float_as_uint(x[3]));
  } else {
    uint2 w;
    w.x = static_cast<uint32_t>(bf16_from_float(x[0])) | (static_cast<uint32_t>(bf16_from_float(x[1])) << 16);
    w.y = static_cast<uint32_t>(bf16_from_float(x[2])) | (static_cast<uint32_t>(bf16_from_float(x[3])) << 16);
    *reinterpret_cast<uint2*>(p) = w;
  }
}

template <typename T, typename TB, int NE>
__global__ __launch_bounds__(kPermThreads) void dequant_rows_perm8_fast(int64_t M, int64_t n_cols, int64_t ncv,
                                                                        DequantBooks b,
                                                                        const int32_t* __restrict__ inv,
                                                                        T* __restrict__ out, int64_t ld_out) {
  extern __shared__ unsigned char smem[];
  T* row = reinterpret_cast<T*>(smem);
  uint16_t* src = reinterpret_cast<uint16_t*>(smem + ((n_cols * sizeof(T) + 15) & ~static_cast<int64_t>(15)));
  for (int64_t j = threadIdx.x; j < n_cols; j += kPermThreads) {
    const int32_t sj = inv[j];
    src[j] = (sj >= 0 && sj < n_cols) ? static_cast<uint16_t>(sj) : static_cast<uint16_t>(0xffff);  // 0xffff: zero
  }
  const int64_t vpr = n_cols / 8;
  const int h = threadIdx.x & 1;
  const int pair = threadIdx.x >> 1;
  constexpr int kPairs = kPermThreads / 2;
  constexpr int kStep = kPairs * kUP;
  constexpr int V = 16 / sizeof(T);
  constexpr int NEa = NE > 0 ? NE : 1;
  const TB* Cb = static_cast<const TB*>(b.C[0]);
  const int32_t* qb = b.q[0];
  const int64_t Kb = b.K[0];
  for (int64_t r = blockIdx.x; r < M; r += gridDim.x) {
    for (int64_t g0 = pair; g0 < vpr; g0 += kStep) {
      // codes of the round (the extended codes of its first vector if that one is critical), then
      // every codeword gather of the round at once
      int32_t q[kUP], qe[NEa];
#pragma unroll
      for (int u = 0; u < kUP; ++u) {
        const int64_t g = g0 + kPairs * u;
        const int32_t v = ld_stream_i32(qb + (g < vpr ? r * b.ldq_base + g : 0));
        q[u] = g < vpr ? v : 0;
      }
      const bool crit0 = NE > 0 && g0 < ncv;
#pragma unroll
      for (int e = 0; e < NE; ++e) {
        const int32_t v = b.q[1 + e][crit0 ? r * b.ldq_ext + g0 : 0];
        qe[e] = crit0 ? v : 0;
      }
      float c[kUP][4], ce[NEa][4];
      bool ok[kUP];
#pragma unroll
      for (int u = 0; u < kUP; ++u) {
        ok[u] = q[u] >= 0 && q[u] < Kb;
        load_cw4t<TB>(Cb, ok[u] ? q[u] : 0, h, c[u]);
      }
#pragma unroll
      for (int e = 0; e < NE; ++e) {
        const bool in = qe[e] >= 0 && qe[e] < b.K[1 + e];
        ok[0] = ok[0] && in;  // qe is 0 (in range) for a vector that is not critical
        load_cw4t<float>(static_cast<const float*>(b.C[1 + e]), in ? qe[e] : 0, h, ce[e]);
      }
#pragma unroll
      for (int u = 0; u < kUP; ++u) {
        const int64_t g = g0 + kPairs * u;
        if (u == 0 && crit0) {
          // fp64 sum in book order: the basic codeword, then the extended books
          double v[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) v[t] = 0.0 + static_cast<double>(c[u][t]);
#pragma unroll
          for (int e = 0; e < NE; ++e)
#pragma unroll
            for (int t = 0; t < 4; ++t) v[t] = v[t] + static_cast<double>(ce[e][t]);
#pragma unroll
          for (int t = 0; t < 4; ++t) v[t] = ok[u] ? v[t] : __builtin_nan("");
          if (g < vpr) store4<T, false>(row + g * 8 + 4 * h, v);
        } else {
          float v[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) v[t] = ok[u] ? c[u][t] : __builtin_nanf("");
          if (g < vpr) store4f<T>(row + g * 8 + 4 * h, v);
        }
      }
    }
    __syncthreads();  // the row (and, first time round, the permutation) is in LDS
    T* ro = out + r * ld_out;
    for (int64_t c = threadIdx.x; c < n_cols / V; c += kPermThreads) {
      T seg[V];
#pragma unroll
      for (int u = 0; u < V; ++u) {
        const uint32_t sj = src[c * V + u];
        seg[u] = (sj < static_cast<uint32_t>(n_cols)) ? row[sj] : T(0);
      }
      st_stream(reinterpret_cast<uint4*>(ro) + c, *reinterpret_cast<const uint4*>(seg));
    }
    __syncthreads();  // the row buffer is rewritten by the next row
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
  // d = 8 fast paths: every book, the output and the minuend 16-byte aligned per vector
  bool fast = d == 8 && books.n_full == 1 && out_type != ET_F64;
  for (int e = 0; e < books.n; ++e) fast = fast && (reinterpret_cast<uintptr_t>(books.C[e]) % 16 == 0);
  const int esize = out_type == ET_F32 ? 4 : (out_type == ET_F64 ? 8 : 2);
  fast = fast && (reinterpret_cast<uintptr_t>(out) % 16 == 0) && ((ld_out * esize) % 16 == 0);
  if (fast && minuend) {
    const int msize = min_type == ET_F32 ? 4 : 2;
    fast = (reinterpret_cast<uintptr_t>(minuend) % 16 == 0) && ((ld_min * msize) % 16 == 0);
  }
  if (fast && !inv_perm) {
    const unsigned grid = static_cast<unsigned>(cdiv(2 * nvec, 256));
    const int64_t vpr = n_cols / 8;
#define CRVQ_DQ8(T, TM)                                                                                       \
  hipLaunchKernelGGL((dequant_rows8<T, TM>), dim3(grid), dim3(256), 0, stream, M, vpr, ncv, books,          \
                     static_cast<const TM*>(minuend), ld_min, static_cast<T*>(out), ld_out)
    if (out_type == ET_F32) {
      if (minuend && min_type == ET_BF16) CRVQ_DQ8(float, uint16_t); else CRVQ_DQ8(float, float);
    } else {
      if (minuend && min_type == ET_F32) CRVQ_DQ8(uint16_t, float); else CRVQ_DQ8(uint16_t, uint16_t);
    }
#undef CRVQ_DQ8
    return hipGetLastError();
  }
  const size_t lds8 = ((static_cast<size_t>(n_cols) * esize + 15) & ~static_cast<size_t>(15)) + 2 * n_cols;
  if (fast && inv_perm && n_cols % (16 / esize) == 0 && n_cols < 65535 && lds8 <= 64 * 1024) {
    // Persistent: as many blocks of 512 threads as are resident on the device at once (registers and
    // LDS permitting), each walking rows block, block + grid, ...  Specialised kernel when there are
    // at most kPE extended books, all fp32, and the critical groups of a row lie within the first
    // vector of every lane pair's round.
    bool spec = books.n - 1 <= kPE && ncv <= kPermThreads / 2;
    for (int e = 1; e < books.n; ++e) spec = spec && books.type[e] == ET_F32;
    const void* fn = nullptr;
    const int ne = books.n - 1;
    const bool bf = books.type[0] == ET_BF16;
#define CRVQ_DQP_NE(T, TB)                                                                                      \
  (ne == 0 ? reinterpret_cast<const void*>(dequant_rows_perm8_fast<T, TB, 0>)                                     \
           : ne == 1 ? reinterpret_cast<const void*>(dequant_rows_perm8_fast<T, TB, 1>)                           \
                     : reinterpret_cast<const void*>(dequant_rows_perm8_fast<T, TB, 2>))
    if (spec)
      fn = esize == 4 ? (bf ? CRVQ_DQP_NE(uint32_t, uint16_t) : CRVQ_DQP_NE(uint32_t, float))
                      : (bf ? CRVQ_DQP_NE(uint16_t, uint16_t) : CRVQ_DQP_NE(uint16_t, float));
    else
      fn = esize == 4 ? reinterpret_cast<const void*>(dequant_rows_perm8<uint32_t>)
                      : reinterpret_cast<const void*>(dequant_rows_perm8<uint16_t>);
#undef CRVQ_DQP_NE
    int per_cu = 1, dev = 0, cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kPermThreads, lds8) != hipSuccess || per_cu < 1)
      per_cu = 1;
    if (hipGetDevice(&dev) == hipSuccess) (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int64_t resident = static_cast<int64_t>(per_cu) * (cus > 0 ? cus : 256);
    const int64_t grid = M < resident ? M : resident;
    void* args[] = {&M, &n_cols, const_cast<int64_t*>(&ncv), const_cast<DequantBooks*>(&books),
                    const_cast<int32_t**>(&inv_perm), &out, &ld_out};
    (void)hipGetLastError();
    return hipLaunchKernel(fn, dim3(static_cast<unsigned>(grid)), dim3(kPermThreads), args, lds8, stream);
    return hipGetLastError();
  }
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
