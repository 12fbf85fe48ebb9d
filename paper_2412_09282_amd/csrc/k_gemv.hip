// Matrix-vector product with a CRVQ-quantized layer, y = W_hat x, where W_hat is the additive
// reconstruction in original channel order (Sec. 4.3, Fig. 3 right of the paper): the stored
// layer is the reordered matrix R (R[:, k] = W_hat[:, perm[k]]) as 8-bit codes, so
//   y_r = sum_k R[r, k] x[perm[k]] = sum_g C_base[q_base[r, g]] . xs_g
//         + sum_{g < n_crit/8} sum_e C_e[q_e[r, g]] . xs_g,       xs_g = x[perm[8g .. 8g+7]].
//
// Basic book (K <= 256): the columns are cut into slices of S = 16 G groups.  A workgroup owns one
// slice and a range of rows; it stages the slice's xs in LDS and builds the lookup table
// LUT[g][k] = C_base[k] . xs_g (fp32, t ascending; thread k keeps codeword k in registers and sweeps
// the groups) while the code bytes of its first rows are in flight.  Then every row costs, per
// group, one LDS lookup at LUT[g][code]: 16 lanes per row, G consecutive groups per lane (one G-byte
// code load), fp32 sums, a 16-lane butterfly, and one partial per (slice, row).
// Extended books (critical groups only, a few percent of the groups): one more column of workgroups
// in the same launch builds LUT_e[g][k] = C_e[k] . xs_g for the critical groups in LDS (or, if those
// tables are too large, takes direct fp32 dot products), looks up every row's extended codes and
// writes one more partial per row.  Then y_r = fp64 sum of the partials in order, rounded once.
// Every sum has a fixed order: results are deterministic.
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

// Sum over the 16 lanes of a DPP row (every lane ends with the same total, formed in the same
// order in lane 0 each time): xor 1 and xor 2 inside quads, then the half-row and row mirrors.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_mov<0xB1>(v);   // quad_perm(1, 0, 3, 2)
  v += dpp_mov<0x4E>(v);   // quad_perm(2, 3, 0, 1)
  v += dpp_mov<0x141>(v);  // row_half_mirror
  v += dpp_mov<0x140>(v);  // row_mirror
  return v;
}
template <int CTRL>
__device__ __forceinline__ double dpp_mov_d(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_mov_dpp(static_cast<int>(b), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_mov_dpp(static_cast<int>(b >> 32), CTRL, 0xf, 0xf, false);
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
}
__device__ __forceinline__ double row16_sum_d(double v) {
  v += dpp_mov_d<0xB1>(v);
  v += dpp_mov_d<0x4E>(v);
  v += dpp_mov_d<0x141>(v);
  v += dpp_mov_d<0x140>(v);
  return v;
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

// Table entry k of one group: the 8-term fp32 dot product C[k] . xs_g, t ascending.
__device__ __forceinline__ float dot8(const float (&c)[8], const float* xg) {
  const float4 x0 = *reinterpret_cast<const float4*>(xg);
  const float4 x1 = *reinterpret_cast<const float4*>(xg + 4);
  float a = c[0] * x0.x;
  a = fmaf(c[1], x0.y, a);
  a = fmaf(c[2], x0.z, a);
  a = fmaf(c[3], x0.w, a);
  a = fmaf(c[4], x1.x, a);
  a = fmaf(c[5], x1.y, a);
  a = fmaf(c[6], x1.z, a);
  a = fmaf(c[7], x1.w, a);
  return a;
}

template <typename TB>
__device__ __forceinline__ void codeword8(const TB* C, int k, float (&c)[8]) {
  if constexpr (sizeof(TB) == 4) {
    const float4 a = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(C) + k * 8);
    const float4 b = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(C) + k * 8 + 4);
    c[0] = a.x; c[1] = a.y; c[2] = a.z; c[3] = a.w; c[4] = b.x; c[5] = b.y; c[6] = b.z; c[7] = b.w;
  } else {
    const uint4 w = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(C) + k * 8);
    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      c[2 * q] = __uint_as_float(u[q] << 16);
      c[2 * q + 1] = __uint_as_float(u[q] & 0xffff0000u);
    }
  }
}

// Table sweep LUT[g][k] = C[k] . xs_g for g < ng: thread t owns codeword k = t % K (loaded into
// registers beforehand by table_codeword) and the groups t / K, t / K + 512 / K, ...; lanes of a
// wave share g (a broadcast read of xs) and write consecutive entries.  Four groups per iteration so
// their LDS reads overlap.
template <typename TB>
__device__ __forceinline__ bool table_codeword(const TB* C, int K, float (&c)[8]) {
  const int tid = threadIdx.x;
  const bool active = tid / K < kGemvThreads / K;  // threads beyond (512 / K) * K idle
  codeword8(C, active ? tid % K : 0, c);
  return active;
}

__device__ __forceinline__ void table_sweep(const float (&c)[8], bool active, int K, const float* xs, int ng,
                                            float* lut) {
  if (!active) return;
  const int tid = threadIdx.x;
  const int per = kGemvThreads / K;  // groups per sweep (K <= 256: at least 2)
  const int k = tid % K;
  int g = tid / K;
  for (; g + 3 * per < ng; g += 4 * per) {
    const float a0 = dot8(c, xs + g * 8);
    const float a1 = dot8(c, xs + (g + per) * 8);
    const float a2 = dot8(c, xs + (g + 2 * per) * 8);
    const float a3 = dot8(c, xs + (g + 3 * per) * 8);
    lut[g * K + k] = a0;
    lut[(g + per) * K + k] = a1;
    lut[(g + 2 * per) * K + k] = a2;
    lut[(g + 3 * per) * K + k] = a3;
  }
  for (; g < ng; g += per) lut[g * K + k] = dot8(c, xs + g * 8);
}

// One workgroup: slice blockIdx.x (groups s0 .. s0 + S - 1), rows [r0, r1).  LDS: LUT [S][K] fp32,
// xs [S][8] fp32.
template <typename TX, bool LUT>
__device__ void ext_rows(int64_t M, int64_t N, int64_t r0, int64_t r1, int64_t ncv, const GemvExt& ext,
                         const int32_t* __restrict__ perm, const TX* __restrict__ x, unsigned char* smem,
                         float* __restrict__ out);

// EXT: columns of workgroups past the slices take the extended books of pieces of their row ranges
// and write them as one more partial.
template <int G, typename TB, typename TX, int EXT>
__global__ __launch_bounds__(kGemvThreads) void gemv_lut_kernel(int64_t M, int64_t N, const uint8_t* __restrict__ q,
                                                                int64_t ldq, const TB* __restrict__ C, int K,
                                                                const int32_t* __restrict__ perm,
                                                                const TX* __restrict__ x, int64_t rows_per_block,
                                                                int64_t ncv, GemvExt ext, float* __restrict__ part) {
  constexpr int S = 16 * G;
  extern __shared__ unsigned char smem[];
  const int n_slices = static_cast<int>((N / 8 + S - 1) / S);
  if (EXT && static_cast<int>(blockIdx.x) >= n_slices) {  // uniform: the extended-book columns
    // column j of E takes the j-th of E equal pieces (whole steps) of the row range
    const int E = static_cast<int>(gridDim.x) - n_slices;
    const int j = static_cast<int>(blockIdx.x) - n_slices;
    const int64_t per = (rows_per_block + E - 1) / E;
    const int64_t piece = (per + kRowsPerStep - 1) / kRowsPerStep * kRowsPerStep;
    const int64_t rr = static_cast<int64_t>(blockIdx.y) * rows_per_block;
    const int64_t rend = (rr + rows_per_block < M) ? rr + rows_per_block : M;
    const int64_t r0 = rr + j * piece;
    const int64_t r1 = (r0 + piece < rend) ? r0 + piece : rend;
    float* out = part + static_cast<int64_t>(n_slices) * M;
    if (EXT == 1)
      ext_rows<TX, true>(M, N, r0, r1, ncv, ext, perm, x, smem, out);
    else
      ext_rows<TX, false>(M, N, r0, r1, ncv, ext, perm, x, smem, out);
    return;
  }
  float* lut = reinterpret_cast<float*>(smem);
  float* xs = lut + S * K;
  const int tid = threadIdx.x;
  const int64_t groups = N / 8;
  const int64_t s0 = static_cast<int64_t>(blockIdx.x) * S;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * rows_per_block;
  const int64_t r1 = (r0 + rows_per_block < M) ? r0 + rows_per_block : M;
  const int sub = tid & 15;  // lane within the row's 16
  const int rs = tid >> 4;   // row slot of the step
  const int64_t g0 = s0 + static_cast<int64_t>(sub) * G;  // first group of this lane
  const bool lane_live = g0 < groups;  // groups / G chunks are whole (N is a multiple of 8 G)

  // Loads in the order their data are needed (the memory counter completes in order): the xs column
  // indices, then the xs gather and the thread's codeword, then the code bytes of the first kPrefetch
  // steps (in flight while the table is built).  Straight-line code: absent entries read index 0.
  constexpr int kXs = (S * 8 + kGemvThreads - 1) / kGemvThreads;  // xs elements per thread
  int64_t src[kXs];
  bool xok[kXs];
#pragma unroll
  for (int i = 0; i < kXs; ++i) {
    const int64_t col = s0 * 8 + tid + i * kGemvThreads;
    xok[i] = tid + i * kGemvThreads < S * 8 && col < N;
    src[i] = xok[i] ? col : 0;
  }
  if (perm) {
#pragma unroll
    for (int i = 0; i < kXs; ++i) src[i] = perm[src[i]];
  }
  float xv[kXs];
#pragma unroll
  for (int i = 0; i < kXs; ++i) {
    const bool in = src[i] >= 0 && src[i] < N;
    const float v = elem_f(x, in ? src[i] : 0);
    xv[i] = !xok[i] ? 0.0f : (in ? v : __builtin_nanf(""));
  }
  float cw[8];
  const bool tab_active = table_codeword(C, K, cw);
  CodeChunk<G> qc[kPrefetch];
  auto load_step = [&](int64_t r, CodeChunk<G>& c) {
    const bool ok = lane_live && r < r1;
    c.load(q + (ok ? r * ldq + g0 : 0));
  };
#pragma unroll
  for (int u = 0; u < kPrefetch; ++u) load_step(r0 + static_cast<int64_t>(u) * kRowsPerStep + rs, qc[u]);
#pragma unroll
  for (int i = 0; i < kXs; ++i)
    if (tid + i * kGemvThreads < S * 8) xs[tid + i * kGemvThreads] = xv[i];
  __syncthreads();
  table_sweep(cw, tab_active, K, xs, static_cast<int>(groups - s0 < S ? groups - s0 : S), lut);
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
      // refill the slot with the step kPrefetch further on (if the workgroup has one)
      if (rb + static_cast<int64_t>(kPrefetch) * kRowsPerStep < r1)
        load_step(r + static_cast<int64_t>(kPrefetch) * kRowsPerStep, qc[u]);
      acc = row16_sum(acc);
      if (sub == 0 && r < r1) pout[r] = acc;
    }
  }
}

// Extended books on the critical groups, rows [r0, r1): out[r] = sum over the books (in order) and the
// row's critical groups of C_e[q_e[r, g]] . xs_g, fp32.  16 lanes per row, 32 rows per step, batches
// of kExtSteps steps whose code bytes are loaded first.  LUT = true: LUT_e[g][k] = C_e[k] . xs_g for
// the critical groups is built in LDS (books in order) and the codes are looked up; otherwise (tables
// too large) each lane takes fp32 dot products with the codewords from memory.
constexpr int kExtSteps = 4;

template <typename TX, bool LUT>
__device__ void ext_rows(int64_t M, int64_t N, int64_t r0, int64_t r1, int64_t ncv, const GemvExt& ext,
                         const int32_t* __restrict__ perm, const TX* __restrict__ x, unsigned char* smem,
                         float* __restrict__ out) {
  const int tid = threadIdx.x;
  const int sub = tid & 15;
  const int rs = tid >> 4;
  float* xs = reinterpret_cast<float*>(smem);  // [ncv][8] when LUT
  float* elut = xs + (LUT ? ncv * 8 : 0);
  if (LUT) {
    // every book's codeword of this thread (first kEarly books) in flight together with the xs loads
    constexpr int kEarly = 3;
    float cw[kEarly][8];
    bool act[kEarly];
#pragma unroll
    for (int e = 0; e < kEarly; ++e) {
      act[e] = false;
      if (e < ext.n) {
        if (ext.type[e] == ET_F32)
          act[e] = table_codeword(static_cast<const float*>(ext.C[e]), ext.K[e], cw[e]);
        else
          act[e] = table_codeword(static_cast<const uint16_t*>(ext.C[e]), ext.K[e], cw[e]);
      }
    }
    for (int64_t e = tid; e < ncv * 8; e += kGemvThreads) {
      const int64_t src = perm ? static_cast<int64_t>(perm[e]) : e;
      xs[e] = (src >= 0 && src < N) ? elem_f(x, src) : __builtin_nanf("");
    }
    __syncthreads();
    int off = 0;
    for (int e = 0; e < ext.n; ++e) {
      float c[8];
      bool a;
      if (e < kEarly) {
#pragma unroll
        for (int t = 0; t < 8; ++t) c[t] = cw[e < kEarly ? e : 0][t];
        a = act[e < kEarly ? e : 0];
      } else if (ext.type[e] == ET_F32) {
        a = table_codeword(static_cast<const float*>(ext.C[e]), ext.K[e], c);
      } else {
        a = table_codeword(static_cast<const uint16_t*>(ext.C[e]), ext.K[e], c);
      }
      table_sweep(c, a, ext.K[e], xs, static_cast<int>(ncv), elut + off);
      off += static_cast<int>(ncv) * ext.K[e];
    }
    __syncthreads();
  }
  // the lane's (book, group) pairs: book e, groups sub, sub + 16, ... below ncv; with at most
  // kMaxPairs of them their code bytes for a batch of steps are loaded before they are used
  constexpr int kMaxPairs = 8;
  const int per_e = static_cast<int>((ncv - sub + 15) / 16 > 0 ? (ncv - sub + 15) / 16 : 0);  // groups of this lane
  const int n_pairs = ext.n * per_e;
  const bool few = n_pairs <= kMaxPairs;
  for (int64_t rb = r0; rb < r1; rb += static_cast<int64_t>(kExtSteps) * kRowsPerStep) {
    uint8_t cq[kExtSteps][kMaxPairs];
    if (LUT && few) {
#pragma unroll
      for (int u = 0; u < kExtSteps; ++u) {
        const int64_t r = rb + u * kRowsPerStep + rs;
#pragma unroll
        for (int pp = 0; pp < kMaxPairs; ++pp) {
          const bool ok = r < r1 && pp < n_pairs;
          const int e = ok ? pp / per_e : 0;
          const int64_t g = sub + 16 * static_cast<int64_t>(ok ? pp - e * per_e : 0);
          cq[u][pp] = ok ? ext.q[e][r * ext.ldq + g] : static_cast<uint8_t>(0);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kExtSteps; ++u) {
      const int64_t r = rb + u * kRowsPerStep + rs;
      float ea = 0.0f;
      bool bad = false;
      if (LUT && few && r < r1) {
        int off = 0, e_prev = 0;
#pragma unroll
        for (int pp = 0; pp < kMaxPairs; ++pp) {
          if (pp < n_pairs) {
            const int e = pp / per_e;
            for (; e_prev < e; ++e_prev) off += static_cast<int>(ncv) * ext.K[e_prev];
            const int64_t g = sub + 16 * static_cast<int64_t>(pp - e * per_e);
            const int Ke = ext.K[e];
            const int code = cq[u][pp];
            bad = bad || code >= Ke;
            ea += elut[off + g * Ke + (code < Ke ? code : 0)];
          }
        }
      } else if (r < r1) {
        int off = 0;
        for (int e = 0; e < ext.n; ++e) {
          const int Ke = ext.K[e];
          for (int64_t g = sub; g < ncv; g += 16) {
            const int code = ext.q[e][r * ext.ldq + g];
            const bool in = code < Ke;
            bad = bad || !in;
            const int k = in ? code : 0;
            if (LUT) {
              ea += elut[off + g * Ke + k];
            } else {
              float xv[8];
#pragma unroll
              for (int t = 0; t < 8; ++t) {
                const int64_t col = g * 8 + t;
                const int64_t src = perm ? static_cast<int64_t>(perm[col]) : col;
                const bool ok = src >= 0 && src < N;
                bad = bad || !ok;
                xv[t] = ok ? elem_f(x, src) : 0.0f;
              }
              float c[8];
              if (ext.type[e] == ET_F32)
                codeword8(static_cast<const float*>(ext.C[e]), k, c);
              else
                codeword8(static_cast<const uint16_t*>(ext.C[e]), k, c);
              float a = c[0] * xv[0];
#pragma unroll
              for (int t = 1; t < 8; ++t) a = fmaf(c[t], xv[t], a);
              ea += a;
            }
          }
          off += static_cast<int>(ncv) * Ke;
        }
      }
      if (bad) ea = __builtin_nanf("");
      ea = row16_sum(ea);
      if (sub == 0 && r < r1) out[r] = ea;
    }
  }
  (void)M;
}

// Finish: y_r = fp64 sum of the partials [0, n_part) in order, rounded once.
__global__ __launch_bounds__(256) void gemv_reduce_kernel(int64_t M, int n_part, const float* __restrict__ part,
                                                          float* __restrict__ y) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (r >= M) return;
  double acc = 0.0;
  for (int s = 0; s < n_part; ++s) acc += static_cast<double>(part[static_cast<int64_t>(s) * M + r]);
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

GemvPlan plan_gemv(int64_t M, int64_t N, int K_base, int64_t ncv, int ext_K_sum, int n_ext) {
  GemvPlan p;
  // the largest slice (16 G groups) whose table and xs fit in the LDS of a CU
  p.G = 8;
  while (p.G > 1 && static_cast<size_t>(16 * p.G) * (K_base * 4 + 32) > static_cast<size_t>(156 * 1024)) p.G >>= 1;
  const int64_t S = 16 * p.G;
  p.n_slices = static_cast<int>(cdiv(N / 8, S));
  p.lds = static_cast<size_t>(S) * (K_base * 4 + 32);
  // extended tables of the critical groups in the finishing kernel when they fit in 96 KiB
  p.ext_lds = static_cast<size_t>(ncv) * 32 + static_cast<size_t>(ncv) * ext_K_sum * 4;
  p.fused = (ext_K_sum > 0 && ncv > 0 && p.ext_lds <= static_cast<size_t>(96 * 1024)) ? 1 : 0;
  // as many workgroups as are resident at once (one per CU when the table needs more than half of
  // the LDS), counting the extended-book column, whole steps of rows per workgroup
  const int64_t resident = p.lds > 78 * 1024 ? 256 : 512;
  // extended-book columns: a lane's (book, group) pairs each cost several slice lookups (a separate
  // byte load each), so a row range gets ceil(3 pairs / 4) columns of them (at most 4) to one per
  // slice
  p.ext_cols = 0;
  if (ext_K_sum > 0 && ncv > 0) {
    const int64_t pairs = static_cast<int64_t>(n_ext) * ((ncv + 15) / 16);
    p.ext_cols = static_cast<int>((3 * pairs + 3) / 4);
    p.ext_cols = p.ext_cols < 1 ? 1 : (p.ext_cols > 4 ? 4 : p.ext_cols);
  }
  const int64_t cols = p.n_slices + p.ext_cols;
  int64_t rb = resident / cols > 0 ? resident / cols : 1;
  const int64_t max_rb = cdiv(M, kRowsPerStep);
  if (rb > max_rb) rb = max_rb;
  if (rb < 1) rb = 1;
  p.rows_per_block = cdiv(cdiv(M, rb), kRowsPerStep) * kRowsPerStep;
  p.row_blocks = cdiv(M, p.rows_per_block);
  return p;
}

size_t gemv_ws_bytes(int64_t M, int64_t N, int K_base) {
  const GemvPlan p = plan_gemv(M, N, K_base, 0, 0, 0);
  return align256(static_cast<size_t>(p.n_slices + 1) * M * 4);  // slices and the extended books
}

hipError_t launch_gemv(int64_t M, int64_t N, int64_t n_crit, const uint8_t* q_base, int64_t ldq_base, const void* C_base,
                       int base_type, int K_base, const GemvExt& ext, const int32_t* perm, const void* x, int x_type,
                       float* y, void* ws, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  const int64_t ncv = n_crit / 8;
  const bool has_ext = ext.n > 0 && ncv > 0;
  int ext_K_sum = 0;
  for (int e = 0; e < ext.n; ++e) ext_K_sum += ext.K[e];
  const GemvPlan p = plan_gemv(M, N, K_base, has_ext ? ncv : 0, has_ext ? ext_K_sum : 0, has_ext ? ext.n : 0);
  float* part = static_cast<float*>(ws);
  const int n_part = p.n_slices + (has_ext ? 1 : 0);
  const dim3 grid(static_cast<unsigned>(p.n_slices + p.ext_cols), static_cast<unsigned>(p.row_blocks));
  const size_t lds = (has_ext && p.fused && p.ext_lds > p.lds) ? p.ext_lds : p.lds;
  const int ext_mode = has_ext ? (p.fused ? 1 : 2) : 0;
#define CRVQ_GEMV_L(G, TB, TX, E)                                                                                \
  hipLaunchKernelGGL((gemv_lut_kernel<G, TB, TX, E>), grid, dim3(kGemvThreads), lds, stream, M, N, q_base, ldq_base, \
                     static_cast<const TB*>(C_base), K_base, perm, static_cast<const TX*>(x), p.rows_per_block, ncv,  \
                     ext, part)
#define CRVQ_GEMV_E(G, TB, TX)                                                  \
  do {                                                                          \
    if (ext_mode == 0) CRVQ_GEMV_L(G, TB, TX, 0);                               \
    else if (ext_mode == 1) CRVQ_GEMV_L(G, TB, TX, 1);                          \
    else CRVQ_GEMV_L(G, TB, TX, 2);                                             \
  } while (0)
#define CRVQ_GEMV_G(TB, TX)                                                         \
  do {                                                                              \
    if (p.G == 8) CRVQ_GEMV_E(8, TB, TX);                                           \
    else if (p.G == 4) CRVQ_GEMV_E(4, TB, TX);                                      \
    else if (p.G == 2) CRVQ_GEMV_E(2, TB, TX);                                      \
    else CRVQ_GEMV_E(1, TB, TX);                                                    \
  } while (0)
  if (base_type == ET_F32) {
    if (x_type == ET_F32) CRVQ_GEMV_G(float, float); else CRVQ_GEMV_G(float, uint16_t);
  } else {
    if (x_type == ET_F32) CRVQ_GEMV_G(uint16_t, float); else CRVQ_GEMV_G(uint16_t, uint16_t);
  }
#undef CRVQ_GEMV_G
#undef CRVQ_GEMV_E
#undef CRVQ_GEMV_L
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(gemv_reduce_kernel, dim3(static_cast<unsigned>(cdiv(M, 256))), dim3(256), 0, stream, M, n_part,
                     part, y);
  return hipGetLastError();
}

}  // namespace crvq
