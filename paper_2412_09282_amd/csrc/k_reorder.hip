// Channel reordering (Sec. 4.2 of the paper, Alg. 1 ReorderChannels), its reverse (Sec. 4.3,
// Fig. 3 right) and the row gathers that move columns and vectors.
//
// rank_perm: perm = stable descending order of the importance (NaN last, equal values by
//   ascending channel).  Each thread owns one channel and counts the channels that precede it; the
//   count is split over up to 64 chunks of the importance array (grid y), each streamed through LDS,
//   and the partial counts are summed in a second pass.  The rank is exact and unique, so
//   perm[rank] = channel is a permutation without any atomic.  N is at most a few ten thousand
//   channels, so the O(N^2) comparisons take microseconds.
// gather_columns: out[r, k] = in[r, src[k]] with the row staged in LDS (coalesced in and out);
//   rows too long for LDS fall back to direct gathers.
#include "crvq_internal.h"

namespace crvq {
namespace {

// The reorder's order as one unsigned 64-bit key: larger importance first, equal importances (and
// -0 / +0) by channel, every NaN after every number and NaNs by channel.  The high word orders -v,
// the low word is the channel.
__device__ __forceinline__ uint64_t rank_key(float v, int64_t i) {
  uint32_t hi;
  if (v != v) {
    hi = 0xffffffffu;
  } else {
    const float f = (v == 0.0f) ? 0.0f : -v;
    const uint32_t u = __float_as_uint(f);
    hi = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  }
  return (static_cast<uint64_t>(hi) << 32) | static_cast<uint32_t>(i);
}

// Partial ranks: block (x, y) counts, for 256 channels, the channels of chunk y that precede them
// (keys compared as integers, staged in LDS).
__global__ __launch_bounds__(256) void rank_partial_kernel(const float* __restrict__ imp, int64_t N, int64_t chunk,
                                                           int32_t* __restrict__ part) {
  __shared__ uint64_t tile[1024];
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const uint64_t kj = rank_key((j < N) ? imp[j] : 0.0f, j);
  const int64_t i0 = static_cast<int64_t>(blockIdx.y) * chunk;
  const int64_t i1 = (i0 + chunk < N) ? i0 + chunk : N;
  int rank = 0;
  for (int64_t base = i0; base < i1; base += 1024) {
    // past the chunk: the largest key, which precedes nothing
    for (int t = threadIdx.x; t < 1024; t += 256)
      tile[t] = (base + t < i1) ? rank_key(imp[base + t], base + t) : ~uint64_t{0};
    __syncthreads();
    const int lim = static_cast<int>((i1 - base) < 1024 ? (i1 - base) : 1024);
    const int lim8 = (lim + 7) & ~7;  // the padding keys are never below kj
#pragma unroll 8
    for (int t = 0; t < lim8; ++t) rank += (tile[t] < kj) ? 1 : 0;
    __syncthreads();
  }
  if (j < N) part[static_cast<int64_t>(blockIdx.y) * N + j] = rank;
}

// rank = sum of the partial ranks; perm[rank] = channel (ranks are distinct, so no two threads collide)
__global__ __launch_bounds__(256) void rank_scatter_kernel(const int32_t* __restrict__ part, int chunks, int64_t N,
                                                           int32_t* __restrict__ perm) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (j >= N) return;
  int64_t rank = 0;
  for (int s = 0; s < chunks; ++s) rank += part[static_cast<int64_t>(s) * N + j];
  if (rank >= 0 && rank < N) perm[rank] = static_cast<int32_t>(j);
}

__global__ __launch_bounds__(256) void fill_i32(int32_t* __restrict__ p, int64_t n, int32_t v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ __launch_bounds__(256) void inverse_perm_kernel(const int32_t* __restrict__ perm, int64_t N,
                                                           int32_t* __restrict__ inv) {
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (k >= N) return;
  const int32_t p = perm[k];
  if (p >= 0 && p < N) inv[p] = static_cast<int32_t>(k);
}

template <typename T>
__global__ __launch_bounds__(256) void gather_cols_lds(const T* __restrict__ in, int64_t ld_in, T* __restrict__ out,
                                                       int64_t ld_out, int64_t N, const int32_t* __restrict__ src) {
  extern __shared__ unsigned char smem[];
  T* row = reinterpret_cast<T*>(smem);
  const int64_t r = blockIdx.x;
  const T* ri = in + r * ld_in;
  for (int64_t c = threadIdx.x; c < N; c += 256) row[c] = ri[c];
  __syncthreads();
  T* ro = out + r * ld_out;
  for (int64_t k = threadIdx.x; k < N; k += 256) {
    const int32_t s = src[k];
    if (s >= 0 && s < N) ro[k] = row[s];
  }
}

// Same with 16-byte row segments (V = 16 / sizeof(T) elements): rows are read and written as uint4,
// sources as int4.  Needs N % V == 0 and 16-byte aligned row starts (checked by the launcher).
template <typename T>
__global__ __launch_bounds__(256) void gather_cols_lds_v(const T* __restrict__ in, int64_t ld_in, T* __restrict__ out,
                                                         int64_t ld_out, int64_t N, const int32_t* __restrict__ src) {
  constexpr int V = 16 / sizeof(T);
  extern __shared__ unsigned char smem[];
  T* row = reinterpret_cast<T*>(smem);
  const int64_t r = blockIdx.x;
  const uint4* ri = reinterpret_cast<const uint4*>(in + r * ld_in);
  const int64_t nv = N / V;
  constexpr int U = 4;  // segments in flight per thread
  for (int64_t c0 = threadIdx.x; c0 < nv; c0 += 256 * U) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = (c0 + u * 256 < nv) ? ld_stream(ri + c0 + u * 256) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (c0 + u * 256 < nv) reinterpret_cast<uint4*>(row)[c0 + u * 256] = v[u];
  }
  __syncthreads();
  uint4* ro = reinterpret_cast<uint4*>(out + r * ld_out);
  for (int64_t c = threadIdx.x; c < nv; c += 256) {
    T seg[V];
#pragma unroll
    for (int q = 0; q < V; q += 4) {
      const int4 s4 = reinterpret_cast<const int4*>(src)[(c * V + q) / 4];
      const int32_t s[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) seg[q + u] = (s[u] >= 0 && s[u] < N) ? row[s[u]] : T(0);
    }
    st_stream(ro + c, *reinterpret_cast<const uint4*>(seg));
  }
}

template <typename T>
__global__ __launch_bounds__(256) void gather_cols_direct(const T* __restrict__ in, int64_t ld_in, T* __restrict__ out,
                                                          int64_t ld_out, int64_t M, int64_t N,
                                                          const int32_t* __restrict__ src) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= M * N) return;
  const int64_t r = e / N;
  const int64_t k = e - r * N;
  const int32_t s = src[k];
  if (s >= 0 && s < N) out[r * ld_out + k] = in[r * ld_in + s];
}

__device__ __forceinline__ int64_t vec_offset(const RowSrc& s, int64_t i) {
  if (s.ld == s.vpr * s.d) return i * s.d;  // rows packed back to back
  const uint32_t r = static_cast<uint32_t>(i) / static_cast<uint32_t>(s.vpr);
  const uint32_t g = static_cast<uint32_t>(i) - r * static_cast<uint32_t>(s.vpr);
  return static_cast<int64_t>(r) * s.ld + static_cast<int64_t>(g) * s.d;
}

__global__ __launch_bounds__(256) void gather_vectors_kernel(RowSrc src, const int64_t* __restrict__ idx, int64_t count,
                                                             void* __restrict__ out, int out_type) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int d = src.d;
  if (e >= count * d) return;
  const int64_t k = e / d;
  const int t = static_cast<int>(e - k * d);
  const int64_t v = idx[k];
  const bool ok = v >= 0 && v < src.n;
  if (src.type == ET_F32) {
    const float x = ok ? static_cast<const float*>(src.base)[vec_offset(src, v) + t] : __builtin_nanf("");
    static_cast<float*>(out)[e] = x;
  } else {
    const uint16_t h = ok ? static_cast<const uint16_t*>(src.base)[vec_offset(src, v) + t] : static_cast<uint16_t>(0x7fc0);
    if (out_type == ET_BF16)
      static_cast<uint16_t*>(out)[e] = h;
    else
      static_cast<float*>(out)[e] = __uint_as_float(static_cast<uint32_t>(h) << 16);
  }
}

}  // namespace

int rank_chunks(int64_t N) {
  const int64_t c = cdiv(N, 256);
  return static_cast<int>(c < 1 ? 1 : (c > 64 ? 64 : c));
}

hipError_t launch_rank_perm(const float* importance, int64_t N, int32_t* perm, int32_t* part, hipStream_t stream) {
  const int S = rank_chunks(N);
  const int64_t chunk = cdiv(N, S);
  hipLaunchKernelGGL(rank_partial_kernel, dim3(static_cast<unsigned>(cdiv(N, 256)), static_cast<unsigned>(S)), dim3(256),
                     0, stream, importance, N, chunk, part);
  hipLaunchKernelGGL(rank_scatter_kernel, dim3(static_cast<unsigned>(cdiv(N, 256))), dim3(256), 0, stream, part, S, N,
                     perm);
  return hipGetLastError();
}

hipError_t launch_inverse_perm(const int32_t* perm, int64_t N, int32_t* inv, hipStream_t stream) {
  const unsigned g = static_cast<unsigned>(cdiv(N, 256));
  hipLaunchKernelGGL(fill_i32, dim3(g), dim3(256), 0, stream, inv, N, -1);
  hipLaunchKernelGGL(inverse_perm_kernel, dim3(g), dim3(256), 0, stream, perm, N, inv);
  return hipGetLastError();
}

hipError_t launch_gather_columns(const void* in, int64_t ld_in, void* out, int64_t ld_out, int esize, int64_t M,
                                 int64_t N, const int32_t* src_idx, hipStream_t stream) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const size_t lds = static_cast<size_t>(N) * esize;
  const int V = 16 / esize;
  const bool vec_ok = (N % V == 0) && ((ld_in * esize) % 16 == 0) && ((ld_out * esize) % 16 == 0) &&
                      (reinterpret_cast<uintptr_t>(in) % 16 == 0) && (reinterpret_cast<uintptr_t>(out) % 16 == 0) &&
                      (reinterpret_cast<uintptr_t>(src_idx) % 16 == 0);
  if (lds <= 64 * 1024 && vec_ok) {
    if (esize == 4)
      hipLaunchKernelGGL(gather_cols_lds_v<uint32_t>, dim3(static_cast<unsigned>(M)), dim3(256), lds, stream,
                         static_cast<const uint32_t*>(in), ld_in, static_cast<uint32_t*>(out), ld_out, N, src_idx);
    else
      hipLaunchKernelGGL(gather_cols_lds_v<uint16_t>, dim3(static_cast<unsigned>(M)), dim3(256), lds, stream,
                         static_cast<const uint16_t*>(in), ld_in, static_cast<uint16_t*>(out), ld_out, N, src_idx);
  } else if (lds <= 64 * 1024) {
    if (esize == 4)
      hipLaunchKernelGGL(gather_cols_lds<uint32_t>, dim3(static_cast<unsigned>(M)), dim3(256), lds, stream,
                         static_cast<const uint32_t*>(in), ld_in, static_cast<uint32_t*>(out), ld_out, N, src_idx);
    else
      hipLaunchKernelGGL(gather_cols_lds<uint16_t>, dim3(static_cast<unsigned>(M)), dim3(256), lds, stream,
                         static_cast<const uint16_t*>(in), ld_in, static_cast<uint16_t*>(out), ld_out, N, src_idx);
  } else {
    dim3 grid(static_cast<unsigned>(cdiv(M * N, 256)));
    if (esize == 4)
      hipLaunchKernelGGL(gather_cols_direct<uint32_t>, grid, dim3(256), 0, stream, static_cast<const uint32_t*>(in), ld_in,
                         static_cast<uint32_t*>(out), ld_out, M, N, src_idx);
    else
      hipLaunchKernelGGL(gather_cols_direct<uint16_t>, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(in), ld_in,
                         static_cast<uint16_t*>(out), ld_out, M, N, src_idx);
  }
  return hipGetLastError();
}

hipError_t launch_gather_vectors(const RowSrc& src, const int64_t* idx, int64_t count, void* out, int out_type,
                                 hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_vectors_kernel, dim3(static_cast<unsigned>(cdiv(count * src.d, 256))), dim3(256), 0, stream,
                     src, idx, count, out, out_type);
  return hipGetLastError();
}

}  // namespace crvq
