// Matrix-vector product with a CRVQ-quantized layer, y = W_hat x, where W_hat is the additive
// reconstruction in original channel order (Sec. 4.3, Fig. 3 right of the paper): the stored
// layer is the reordered matrix R (R[:, k] = W_hat[:, perm[k]]) as 8-bit codes, so
//   y_r = sum_k R[r, k] x[perm[k]] = sum_g C_base[q_base[r, g]] . xs_g
//         + sum_{g < n_crit/8} sum_e C_e[q_e[r, g]] . xs_g,       xs_g = x[perm[8g .. 8g+7]].
//
// Basic book (K <= 256): the columns are cut into slices of S = 16 G groups.  A workgroup owns one
// slice and a range of rows; it stages the slice's xs and the codebook in LDS and builds the
// lookup table LUT[g][k] = C_base[k] . xs_g (fp32, t ascending) for the slice, with the code bytes
// of its first rows already in flight.  Then every row costs, per group, one LDS lookup at
// LUT[g][code]: 16 lanes per row, G consecutive groups per lane (one G-byte code load), fp32 sums,
// a 16-lane butterfly, and one partial per (slice, row).
// Extended books (critical groups only, a few percent of the groups): a direct fp32 dot product of
// the codewords with xs per critical group, one partial per row.
// Reduction: y_r = fp64 sum of the slice partials in slice order plus the extended partial, rounded
// once.  Every sum has a fixed order: results are deterministic.
#include "crvq_internal.h"

namespace crvq {
namespace {

constexpr int kGemvThreads = 512;  // 8 waves, 4 rows of 16 lanes each per wave and step
constexpr int kRowsPerStep = kGemvThreads / 16;
constexpr int kPrefetch = 8;  // steps whose code bytes are loaded at once

template <typename T>
__device__ __forceinline__ float elem_f(const T* p, int64_t i) {
  if constexpr (sizeof(T) == 4)
    return static_cast<const float*>(static_cast<const void*>(p))[i];
  else
    return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}

// G code bytes of one lane (G in {1, 2, 4, 8}); the load is G bytes wide and G-byte aligned.
template <int G>
struct CodeChunk;
template <>
struct CodeChunk<8> {
  uint64_t v;
  __device__ __forceinline__ void load(const uint8_t* p) { v = __builtin_nontemporal_load(reinterpret_cast<const uint64_t*>(p)); }
  __device__ __forceinline__ int at(int j) const { return static_cast<int>((v >> (8 * j)) & 255); }
};
template <>
struct CodeChunk<4> {
  uint32_t v;
  __device__ __forceinline__ void load(const uint8_t* p) { v = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p)); }
  __device__ __forceinline__ int at(int j) const { return (v >> (8 * j)) & 255; }
};
template <>
struct CodeChunk<2> {
  uint16_t v;
  __device__ __forceinline__ void load(const uint8_t* p) { v = __builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(p)); }
  __device__ __forceinline__ int at(int j) const { return (v >> (8 * j)) & 255; }
};
template <>
struct CodeChunk<1> {
  uint8_t v;
  __device__ __forceinline__ void load(const uint8_t* p) { v = __builtin_nontemporal_load(p); }
  __device__ __forceinline__ int at(int) const { return v; }
};

// One workgroup: slice blockIdx.x (groups s0 .. s0 + S - 1), rows [r0, r1).
// LDS: LUT [S][K] fp32, codebook [K][8] fp32, xs [S][8] fp32.
template <int G, typename TB, typename TX>
__global__ __launch_bounds__(kGemvThreads) void gemv_lut_kernel(int64_t M, int64_t N, const uint8_t* __restrict__ q,
                                                                int64_t ldq, const TB* __restrict__ C, int K,
                                                                const int32_t* __restrict__ perm,
                                                                const TX* __restrict__ x, int64_t rows_per_block,
                                                                float* __restrict__ part) {
  constexpr int S = 16 * G;
  extern __shared__ unsigned char smem[];
  float* lut = reinterpret_cast<float*>(smem);
  float* cb = lut + S * K;
  float* xs = cb + K * 8;
  const int tid = threadIdx.x;
  const int64_t groups = N / 8;
  const int64_t s0 = static_cast<int64_t>(blockIdx.x) * S;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * rows_per_block;
  const int64_t r1 = (r0 + rows_per_block < M) ? r0 + rows_per_block : M;
  const int sub = tid & 15;  // lane within the row's 16
  const int rs = tid >> 4;   // row slot of the step
  const int64_t g0 = s0 + static_cast<int64_t>(sub) * G;  // first group of this lane
  const bool lane_live = g0 < groups;  // groups / G chunks are whole (N is a multiple of 8 G)

  // code bytes of the first kPrefetch steps, in flight while the table is built
  CodeChunk<G> qc[kPrefetch];
  auto load_step = [&](int64_t r, CodeChunk<G>& c) {
    const bool ok = lane_live && r < r1;
    c.load(q + (ok ? r * ldq + g0 : 0));
  };
#pragma unroll
  for (int u = 0; u < kPrefetch; ++u) load_step(r0 + static_cast<int64_t>(u) * kRowsPerStep + rs, qc[u]);

  // stage xs (gathered through perm) and the codebook, then build LUT[g][k]
  for (int e = tid; e < S * 8; e += kGemvThreads) {
    const int64_t col = s0 * 8 + e;
    float v = 0.0f;
    if (col < N) {
      int64_t src = perm ? static_cast<int64_t>(perm[col]) : col;
      v = (src >= 0 && src < N) ? elem_f(x, src) : __builtin_nanf("");
    }
    xs[e] = v;
  }
  for (int e = tid; e < K * 8; e += kGemvThreads) cb[e] = elem_f(C, e);
  __syncthreads();
  for (int e = tid; e < S * K; e += kGemvThreads) {
    const int g = e / K;
    const int k = e - g * K;
    const float4 c0 = *reinterpret_cast<const float4*>(cb + k * 8);
    const float4 c1 = *reinterpret_cast<const float4*>(cb + k * 8 + 4);
    const float4 x0 = *reinterpret_cast<const float4*>(xs + g * 8);
    const float4 x1 = *reinterpret_cast<const float4*>(xs + g * 8 + 4);
    float a = c0.x * x0.x;
    a = fmaf(c0.y, x0.y, a);
    a = fmaf(c0.z, x0.z, a);
    a = fmaf(c0.w, x0.w, a);
    a = fmaf(c1.x, x1.x, a);
    a = fmaf(c1.y, x1.y, a);
    a = fmaf(c1.z, x1.z, a);
    a = fmaf(c1.w, x1.w, a);
    lut[e] = a;
  }
  __syncthreads();

  const float* lrow = lut + static_cast<int64_t>(sub) * G * K;
  float* pout = part + static_cast<int64_t>(blockIdx.x) * M;
  for (int64_t rb = r0; rb < r1; rb += static_cast<int64_t>(kPrefetch) * kRowsPerStep) {
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) {
      const int64_t r = rb + static_cast<int64_t>(u) * kRowsPerStep + rs;
      float acc = 0.0f;
      bool bad = false;
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const int code = qc[u].at(j);
        bad = bad || code >= K;
        acc += lrow[j * K + (code < K ? code : 0)];
      }
      if (!lane_live) acc = 0.0f;
      if (bad && lane_live) acc = __builtin_nanf("");
      // refill the slot with the step kPrefetch further on
      load_step(r + static_cast<int64_t>(kPrefetch) * kRowsPerStep, qc[u]);
#pragma unroll
      for (int m = 8; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 16);
      if (sub == 0 && r < r1) pout[r] = acc;
    }
  }
}

// Extended books on the critical groups: 16 lanes per row, lane takes groups sub, sub + 16, ...
template <typename TX>
__global__ __launch_bounds__(kGemvThreads) void gemv_ext_kernel(int64_t M, int64_t N, int64_t ncv, GemvExt ext,
                                                                const int32_t* __restrict__ perm,
                                                                const TX* __restrict__ x, float* __restrict__ out) {
  const int sub = threadIdx.x & 15;
  const int64_t r = static_cast<int64_t>(blockIdx.x) * kRowsPerStep + (threadIdx.x >> 4);
  float acc = 0.0f;
  bool bad = false;
  if (r < M) {
    for (int64_t g = sub; g < ncv; g += 16) {
      float xv[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int64_t col = g * 8 + t;
        const int64_t src = perm ? static_cast<int64_t>(perm[col]) : col;
        const bool ok = src >= 0 && src < N;
        bad = bad || !ok;
        xv[t] = ok ? elem_f(x, src) : 0.0f;
      }
      for (int e = 0; e < ext.n; ++e) {
        const int code = ext.q[e][r * ext.ldq + g];
        const bool in = code < ext.K[e];
        bad = bad || !in;
        const int64_t k = in ? code : 0;
        float a = 0.0f;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const float c = ext.type[e] == ET_F32 ? static_cast<const float*>(ext.C[e])[k * 8 + t]
                                                : __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(ext.C[e])[k * 8 + t]) << 16);
          a = fmaf(c, xv[t], a);
        }
        acc += a;
      }
    }
  }
  if (bad) acc = __builtin_nanf("");
#pragma unroll
  for (int m = 8; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 16);
  if (sub == 0 && r < M) out[r] = acc;
}

__global__ __launch_bounds__(256) void gemv_reduce_kernel(int64_t M, int n_slices, const float* __restrict__ part,
                                                          const float* __restrict__ ext_part,
                                                          float* __restrict__ y) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (r >= M) return;
  double acc = 0.0;
  for (int s = 0; s < n_slices; ++s) acc += static_cast<double>(part[static_cast<int64_t>(s) * M + r]);
  if (ext_part) acc += static_cast<double>(ext_part[r]);
  y[r] = static_cast<float>(acc);
}

__global__ __launch_bounds__(256) void pack_u8_kernel(const int32_t* __restrict__ codes, int64_t n,
                                                      uint8_t* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) out[i] = static_cast<uint8_t>(codes[i] & 255);
}

}  // namespace

hipError_t launch_pack_codes_u8(const int32_t* codes, int64_t n, uint8_t* out, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(pack_u8_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0, stream, codes, n, out);
  return hipGetLastError();
}

GemvPlan plan_gemv(int64_t M, int64_t N, int K_base) {
  GemvPlan p;
  // the largest slice whose table fits next to the codebook and xs in the LDS of one CU
  p.G = 8;
  while (p.G > 1 && static_cast<size_t>(16 * p.G) * K_base * 4 + static_cast<size_t>(K_base) * 32 + 16 * p.G * 32 >
                        static_cast<size_t>(152 * 1024))
    p.G >>= 1;
  const int64_t S = 16 * p.G;
  p.n_slices = static_cast<int>(cdiv(N / 8, S));
  p.lds = static_cast<size_t>(S) * K_base * 4 + static_cast<size_t>(K_base) * 32 + static_cast<size_t>(S) * 32;
  // as many workgroups as are resident at once (one per CU when the table needs more than half
  // of the LDS), whole steps of rows per workgroup
  const int64_t resident = p.lds > 80 * 1024 ? 256 : 512;
  int64_t rb = cdiv(resident, p.n_slices);
  const int64_t max_rb = cdiv(M, kRowsPerStep);
  if (rb > max_rb) rb = max_rb;
  if (rb < 1) rb = 1;
  p.rows_per_block = cdiv(cdiv(M, rb), kRowsPerStep) * kRowsPerStep;
  p.row_blocks = cdiv(M, p.rows_per_block);
  return p;
}

size_t gemv_ws_bytes(int64_t M, int64_t N, int K_base) {
  const GemvPlan p = plan_gemv(M, N, K_base);
  return align256(static_cast<size_t>(p.n_slices) * M * 4) + align256(static_cast<size_t>(M) * 4);
}

hipError_t launch_gemv(int64_t M, int64_t N, int64_t n_crit, const uint8_t* q_base, int64_t ldq_base, const void* C_base,
                       int base_type, int K_base, const GemvExt& ext, const int32_t* perm, const void* x, int x_type,
                       float* y, void* ws, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  const GemvPlan p = plan_gemv(M, N, K_base);
  float* part = static_cast<float*>(ws);
  float* ext_part = reinterpret_cast<float*>(static_cast<char*>(ws) + align256(static_cast<size_t>(p.n_slices) * M * 4));
  const dim3 grid(static_cast<unsigned>(p.n_slices), static_cast<unsigned>(p.row_blocks));
#define CRVQ_GEMV_L(G, TB, TX)                                                                                    \
  hipLaunchKernelGGL((gemv_lut_kernel<G, TB, TX>), grid, dim3(kGemvThreads), p.lds, stream, M, N, q_base, ldq_base, \
                     static_cast<const TB*>(C_base), K_base, perm, static_cast<const TX*>(x), p.rows_per_block, part)
#define CRVQ_GEMV_G(TB, TX)                                                         \
  do {                                                                              \
    if (p.G == 8) CRVQ_GEMV_L(8, TB, TX);                                           \
    else if (p.G == 4) CRVQ_GEMV_L(4, TB, TX);                                      \
    else if (p.G == 2) CRVQ_GEMV_L(2, TB, TX);                                      \
    else CRVQ_GEMV_L(1, TB, TX);                                                    \
  } while (0)
  if (base_type == ET_F32) {
    if (x_type == ET_F32) CRVQ_GEMV_G(float, float); else CRVQ_GEMV_G(float, uint16_t);
  } else {
    if (x_type == ET_F32) CRVQ_GEMV_G(uint16_t, float); else CRVQ_GEMV_G(uint16_t, uint16_t);
  }
#undef CRVQ_GEMV_G
#undef CRVQ_GEMV_L
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t ncv = n_crit / 8;
  const bool has_ext = ext.n > 0 && ncv > 0;
  if (has_ext) {
    const unsigned eg = static_cast<unsigned>(cdiv(M, kRowsPerStep));
    if (x_type == ET_F32)
      hipLaunchKernelGGL(gemv_ext_kernel<float>, dim3(eg), dim3(kGemvThreads), 0, stream, M, N, ncv, ext, perm,
                         static_cast<const float*>(x), ext_part);
    else
      hipLaunchKernelGGL(gemv_ext_kernel<uint16_t>, dim3(eg), dim3(kGemvThreads), 0, stream, M, N, ncv, ext, perm,
                         static_cast<const uint16_t*>(x), ext_part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(gemv_reduce_kernel, dim3(static_cast<unsigned>(cdiv(M, 256))), dim3(256), 0, stream, M,
                     p.n_slices, part, has_ext ? ext_part : nullptr, y);
  return hipGetLastError();
}

}  // namespace crvq
