// Nearest-codeword search for CRVQ on gfx950 (Sec. 3.1 Eq. 3-4 of the paper; the beam's
// per-parent top-B search of Sec. 3.1 / Alg. 1 BeamSearchOptimize).
//
// Distances are split as ||x - c||^2 = ||x||^2 + s(c),  s(c) = ||c||^2 - 2 x.c.
//
// 1. prep: the codebook is repacked into MFMA A-operand order with ||c||^2 (+inf for padding).
// 2. screen: every wave keeps its rows resident as the MFMA B operand (-2x) and streams all codeword
//    tiles of its codebook split; the lanes reduce the s values they receive to running minima and
//    keep, per row, the best tiles (or chunks of tiles) and the smallest minimum of everything else
//    ("rest").  Nothing of the N x K distance matrix leaves the registers.  Three operand forms:
//    * d <= 8, top-1 over long codebooks: 32 x 32 tiles, operands split into two fp16 terms under a
//      power-of-two codebook scale, two v_mfma_f32_32x32x16_f16 per tile (screen32_kernel);
//    * d <= 8 otherwise: 16 x 16 tiles, operands split into two bf16 terms, one
//      v_mfma_f32_16x16x32_bf16 per tile (SplitOps);
//    * d <= 16: fp32 operands, v_mfma_f32_16x16x4_f32 (F32Ops).
//    Top-1 screens re-score the winning lane group's codewords of the kept tile or chunk exactly in
//    fp64 before leaving; top-B screens hand the kept tile ids to the finalize.
// 3. finalize (one thread per row): merge the codebook splits (top-B: re-score the kept tiles in
//    fp64 in the definition's direct form, sum_t (x_t - c_t)^2 with t ascending) and order by (D, k).
// 4. certify / rescue: with R = ||x|| + sqrt(D_top), every codeword that could beat the kept ones
//    has ||c|| <= R, hence a screen error below delta(R) (accumulation, split remainder, underflow);
//    if rest + ||x||^2 - delta > D_top the kept list is provably the exact answer, otherwise the
//    row is appended to a list that the rescue kernel re-searches exactly over the whole codebook
//    in fp64.  Codes therefore equal the fp64 definition's, ties included.
#include "crvq_internal.h"

#include <climits>

#ifndef CRVQ_MIN_TRACKED_TILES
#define CRVQ_MIN_TRACKED_TILES 1
#endif
#ifndef CRVQ_SCREEN_PREFETCH
#define CRVQ_SCREEN_PREFETCH 1
#endif
#ifndef CRVQ_CB_WIDE
#define CRVQ_CB_WIDE 8  // column blocks per wave for top-1/top-2 screens on large row counts
#endif
#ifndef CRVQ_SPLIT_SCREEN
#define CRVQ_SPLIT_SCREEN 1  // split-bf16 MFMA screen for d <= 8 (0: fp32 MFMA for every d)
#endif
#ifndef CRVQ_CHUNK
#define CRVQ_CHUNK 8  // tiles per tracking chunk of the top-1 screen on long tile ranges
#endif
#ifndef CRVQ_CHUNK_TOPB
#define CRVQ_CHUNK_TOPB 4  // tiles per chunk of the top-B screen (B = 2, 4, 8) on long tile ranges
#endif
#ifndef CRVQ_CHUNK_MIN_TILES
#define CRVQ_CHUNK_MIN_TILES 128  // shorter tile ranges track single tiles (cheaper exact epilogue)
#endif
#ifndef CRVQ_S32_SCREEN
#define CRVQ_S32_SCREEN 1  // 32 x 32 split-fp16 tiles for long top-1 searches
#endif
#ifndef CRVQ_S32_MIN_TILES
#define CRVQ_S32_MIN_TILES 256  // 16-codeword tiles per split from which the 32 x 32 screen is used
#endif
#ifndef CRVQ_S32_CB
#define CRVQ_S32_CB 4  // 32-row column blocks per wave
#endif
#ifndef CRVQ_S32_CHUNK
#define CRVQ_S32_CHUNK 2  // 32-codeword tiles per tracking chunk (1 or 2)
#endif
#ifndef CRVQ_DEBUG_RESCUE
#define CRVQ_DEBUG_RESCUE 0
#endif
#ifndef CRVQ_RESCUE_FILTER
#define CRVQ_RESCUE_FILTER 1  // top-1 rescue: batched rows with a bounded fp32 filter before fp64
#endif
#ifndef CRVQ_S32_SCHED
#define CRVQ_S32_SCHED 1  // pin the MFMA / VALU interleave of the 32 x 32 screen
#endif
#ifndef CRVQ_PRUNE
#define CRVQ_PRUNE 1  // certified chunk skipping in the long top-1 screens (a norm band and two coordinate bands)
#endif
#ifndef CRVQ_PRUNE_FIRST
#define CRVQ_PRUNE_FIRST 4  // chunks screened before the first band; the band is renewed after 2x, 4x, ...
#endif
#ifndef CRVQ_PRUNE2
#define CRVQ_PRUNE2 1  // the second screen after a pruned first one skips chunks too (fixed bands)
#endif
#ifndef CRVQ_PRUNE2_SB
#define CRVQ_PRUNE2_SB 1
#endif
#ifndef CRVQ_PRUNE_CAP
#define CRVQ_PRUNE_CAP 128  // ... and then every this many chunks
#endif

namespace crvq {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

__device__ __forceinline__ int64_t row_offset(const RowSrc& s, int64_t i) {
  if (s.type == ET_F64 || s.ld == s.vpr * s.d) return i * s.d;  // rows packed back to back
  // a column slab: 32-bit division (vector counts are below 2^31)
  const uint32_t r = static_cast<uint32_t>(i) / static_cast<uint32_t>(s.vpr);
  const uint32_t g = static_cast<uint32_t>(i) - r * static_cast<uint32_t>(s.vpr);
  return static_cast<int64_t>(r) * s.ld + static_cast<int64_t>(g) * s.d;
}

__device__ __forceinline__ double row_elem(const RowSrc& s, int64_t off, int t) {
  if (s.type == ET_F32) return static_cast<double>(static_cast<const float*>(s.base)[off + t]);
  if (s.type == ET_BF16) return static_cast<double>(bf16_to_f(static_cast<const uint16_t*>(s.base)[off + t]));
  return static_cast<const double*>(s.base)[off + t];
}

__device__ __forceinline__ double cb_elem(const void* C, int type, int64_t k, int d, int t) {
  if (type == ET_F32) return static_cast<double>(static_cast<const float*>(C)[k * d + t]);
  return static_cast<double>(bf16_to_f(static_cast<const uint16_t*>(C)[k * d + t]));
}

// The first DM elements of row i in fp64 (zero past d or for an invalid row).  The type is
// dispatched once and every load is issued before any is used.
// DM fp32 / bf16 elements at p as floats: 16-byte vector loads when d fills DM and p is aligned
// (every lane then reads one contiguous piece), element loads otherwise; zero past d or when !ok.
template <int DM>
__device__ __forceinline__ void load_f32_elems(const float* p, int d, bool ok, float (&v)[DM]) {
  if (DM % 4 == 0 && d == DM && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
#pragma unroll
    for (int q = 0; q < DM / 4; ++q) {
      const f4 w = ok ? reinterpret_cast<const f4*>(p)[q] : f4{0.0f, 0.0f, 0.0f, 0.0f};
      v[4 * q] = w[0];
      v[4 * q + 1] = w[1];
      v[4 * q + 2] = w[2];
      v[4 * q + 3] = w[3];
    }
  } else {
#pragma unroll
    for (int t = 0; t < DM; ++t) v[t] = (ok && t < d) ? p[t] : 0.0f;
  }
}

template <int DM>
__device__ __forceinline__ void load_bf16_elems(const uint16_t* p, int d, bool ok, float (&v)[DM]) {
  if (DM % 4 == 0 && d == DM && (reinterpret_cast<uintptr_t>(p) & 7) == 0) {
#pragma unroll
    for (int q = 0; q < DM / 4; ++q) {
      const uint2 w = ok ? reinterpret_cast<const uint2*>(p)[q] : make_uint2(0u, 0u);
      v[4 * q] = __uint_as_float(w.x << 16);
      v[4 * q + 1] = __uint_as_float(w.x & 0xffff0000u);
      v[4 * q + 2] = __uint_as_float(w.y << 16);
      v[4 * q + 3] = __uint_as_float(w.y & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int t = 0; t < DM; ++t) v[t] = (ok && t < d) ? bf16_to_f(p[t]) : 0.0f;
  }
}

// The first DM elements of row i in fp64 (zero past d or for an invalid row).  The type is
// dispatched once and every load is issued before any is used.
template <int DM>
__device__ __forceinline__ void load_row_exact(const RowSrc& s, int64_t i, bool valid, double (&x)[DM]) {
  const int d = s.d;
  const int64_t off = valid ? row_offset(s, i) : 0;
  if (s.type == ET_F64) {
    const double* p = static_cast<const double*>(s.base) + off;
#pragma unroll
    for (int t = 0; t < DM; ++t) x[t] = (valid && t < d) ? p[t] : 0.0;
    return;
  }
  float v[DM];
  if (s.type == ET_F32)
    load_f32_elems<DM>(static_cast<const float*>(s.base) + off, d, valid, v);
  else
    load_bf16_elems<DM>(static_cast<const uint16_t*>(s.base) + off, d, valid, v);
#pragma unroll
  for (int t = 0; t < DM; ++t) x[t] = static_cast<double>(v[t]);
}

// Codeword k as float (exact for fp32 and bf16 books), zero past d or when !ok.
template <int DM>
__device__ __forceinline__ void load_codeword(const void* C, int ct, int64_t k, int d, bool ok, float (&c)[DM]) {
  if (ct == ET_F32)
    load_f32_elems<DM>(static_cast<const float*>(C) + (ok ? k * d : 0), d, ok, c);
  else
    load_bf16_elems<DM>(static_cast<const uint16_t*>(C) + (ok ? k * d : 0), d, ok, c);
}

// Appends row i to the list when `fail`, one atomic per wave: the failing lanes of the wave take
// consecutive slots after the wave's leader reserves them.  Every active lane of the wave must call it.
__device__ __forceinline__ void list_append(bool fail, int64_t i, int* rcount, int* rlist) {
  const uint64_t m = __ballot(fail);
  if (m == 0) return;
  const int lane = threadIdx.x & 63;
  const int leader = __ffsll(static_cast<long long>(m)) - 1;
  int base = 0;
  if (lane == leader) base = atomicAdd(rcount, __popcll(m));
  base = __shfl(base, leader);
  if (fail) rlist[base + __popcll(m & ((1ull << lane) - 1ull))] = static_cast<int>(i);
}

__device__ __forceinline__ bool cless(double Da, int ka, double Db, int kb) {
  return Da < Db || (Da == Db && ka < kb);
}

// Insert (D, k) into an ascending list of NB entries, dropping the largest.
template <int NB>
__device__ __forceinline__ void list_insert(double (&LD)[NB], int (&LK)[NB], double D, int k) {
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    bool lt = cless(D, k, LD[j], LK[j]);
    double tD = lt ? LD[j] : D;
    int tk = lt ? LK[j] : k;
    LD[j] = lt ? D : LD[j];
    LK[j] = lt ? k : LK[j];
    D = tD;
    k = tk;
  }
}

// Compare-exchange of two (D, k) pairs: a ends with the (D, k)-smaller.
__device__ __forceinline__ void cswap(double& Da, int& ka, double& Db, int& kb) {
  const bool lt = cless(Db, kb, Da, ka);
  const double lD = lt ? Db : Da, hD = lt ? Da : Db;
  const int lk = lt ? kb : ka, hk = lt ? ka : kb;
  Da = lD;
  ka = lk;
  Db = hD;
  kb = hk;
}

// Four (D, k) candidates into the ascending list of the NB smallest (NB >= 4), the list four calls of
// list_insert would leave: the four are sorted (five compare-exchanges), the last four slots keep the
// smaller of themselves and the candidates taken in reverse (the NB smallest of both, as a bitonic
// sequence), and a half-cleaner network sorts them (about 21 compare-exchanges against 32).
template <int NB>
__device__ __forceinline__ void list_merge4(double (&LD)[NB], int (&LK)[NB], double (&D)[4], int (&Kc)[4]) {
  static_assert(NB >= 4 && (NB & (NB - 1)) == 0, "a power of two of at least four");
  cswap(D[0], Kc[0], D[1], Kc[1]);
  cswap(D[2], Kc[2], D[3], Kc[3]);
  cswap(D[0], Kc[0], D[2], Kc[2]);
  cswap(D[1], Kc[1], D[3], Kc[3]);
  cswap(D[1], Kc[1], D[2], Kc[2]);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int sl = NB - 4 + j;
    const bool take = cless(D[3 - j], Kc[3 - j], LD[sl], LK[sl]);
    LD[sl] = take ? D[3 - j] : LD[sl];
    LK[sl] = take ? Kc[3 - j] : LK[sl];
  }
#pragma unroll
  for (int w = NB / 2; w >= 1; w >>= 1) {
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if ((j & w) == 0) cswap(LD[j], LK[j], LD[j + w], LK[j + w]);
  }
}

// Keep the NB smallest of two ascending lists (bitonic merge; both operands end identical when
// called symmetrically across lanes).
template <int NB>
__device__ __forceinline__ void list_merge(double (&LD)[NB], int (&LK)[NB], const double (&OD)[NB],
                                           const int (&OK)[NB]) {
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    bool take = cless(OD[NB - 1 - j], OK[NB - 1 - j], LD[j], LK[j]);
    LD[j] = take ? OD[NB - 1 - j] : LD[j];
    LK[j] = take ? OK[NB - 1 - j] : LK[j];
  }
#pragma unroll
  for (int s = NB / 2; s >= 1; s /= 2) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if ((j & s) == 0) {
        bool sw = cless(LD[j + s], LK[j + s], LD[j], LK[j]);
        double a = LD[j], b = LD[j + s];
        int ka = LK[j], kb = LK[j + s];
        LD[j] = sw ? b : a;
        LD[j + s] = sw ? a : b;
        LK[j] = sw ? kb : ka;
        LK[j + s] = sw ? ka : kb;
      }
    }
  }
}

template <int NB>
__device__ __forceinline__ void list_merge_xor(double (&LD)[NB], int (&LK)[NB], int mask) {
  double OD[NB];
  int OK[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    OD[j] = __shfl_xor(LD[j], mask);
    OK[j] = __shfl_xor(LK[j], mask);
  }
  list_merge<NB>(LD, LK, OD, OK);
}

// ------------------------------------------------------------------------------------------------
// 1. codebook repack
// ------------------------------------------------------------------------------------------------
// (every prep kernel also clears the rescue counter of the call: thread 0 of block 0)
template <int KS>
__global__ __launch_bounds__(256) void prep_codebook(const void* __restrict__ C, int ct, int64_t K, int d,
                                                     int64_t tiles, float* __restrict__ apack,
                                                     float* __restrict__ cnp, int* __restrict__ rcount) {
  int64_t k = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (k == 0) *rcount = 0;
  if (k >= tiles * 16) return;
  float c[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) c[t] = (k < K && t < d) ? static_cast<float>(cb_elem(C, ct, k, d, t)) : 0.0f;
  float cn = 0.0f;
#pragma unroll
  for (int t = 0; t < 16; ++t) cn = cn + c[t] * c[t];
  cnp[k] = (k < K) ? cn : __builtin_inff();
  const int64_t tile = k >> 4;
  const int i = static_cast<int>(k & 15);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
#pragma unroll
    for (int s = 0; s < KS; ++s) apack[((tile * 64) + i + 16 * q) * KS + s] = c[4 * s + q];
  }
}

template <int KS>
struct AVec;
template <>
struct AVec<1> {
  float v[1];
  __device__ __forceinline__ void load(const float* p) { v[0] = *p; }
};
template <>
struct AVec<2> {
  float v[2];
  __device__ __forceinline__ void load(const float* p) {
    f2 t = *reinterpret_cast<const f2*>(p);
    v[0] = t[0];
    v[1] = t[1];
  }
};
template <>
struct AVec<4> {
  float v[4];
  __device__ __forceinline__ void load(const float* p) {
    f4 t = *reinterpret_cast<const f4*>(p);
    v[0] = t[0];
    v[1] = t[1];
    v[2] = t[2];
    v[3] = t[3];
  }
};

// fp32 to bf16, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t bf16_rn_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Two-term bf16 split of v: hi = bf16(v), lo = bf16(v - hi) (v - hi is exact in fp32), so that
// |v - hi - lo| <= 2^-16 |v|.
__device__ __forceinline__ void bf16_split(float v, uint16_t& hi, uint16_t& lo) {
  hi = bf16_rn_bits(v);
  lo = bf16_rn_bits(v - __uint_as_float(static_cast<uint32_t>(hi) << 16));
}

typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
typedef float f2v __attribute__((ext_vector_type(2)));

// bf16 nearest-even of (a, b), a in the low half: one v_cvt_pk_bf16_f32, which rounds every finite
// fp32 value (subnormals included) to the same bits as bf16_rn_bits.
__device__ __forceinline__ uint32_t bf16x2_rn(float a, float b) {
  const f2v p = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(p, bf2v));
}

// The pair (a, b) of bf16_split: hi terms when !lo_term, else the lo terms.
__device__ __forceinline__ uint32_t bf16x2_split(float a, float b, bool lo_term) {
  const uint32_t h = bf16x2_rn(a, b);
  const uint32_t l = bf16x2_rn(a - __uint_as_float(h << 16), b - __uint_as_float(h & 0xffff0000u));
  return lo_term ? l : h;
}

// Screen operand policies.  Each gives the per-lane A (codebook tile) and B (-2x of the wave's rows)
// operands of one 16 x 16 tile of s values and the MFMA sequence that accumulates them onto ||c||^2.
// Both leave lane l the values of codewords 4 (l / 16) + r, r = 0..3, for row l % 16.
//
// F32Ops: ceil(d / 4) v_mfma_f32_16x16x4_f32 steps; lane l holds dimension 4 s + l / 16 of
//   codeword l % 16 (A) and of row l % 16 (B).
template <int KS>
struct F32Ops {
  static constexpr int DM = 4 * KS;
  struct A {
    AVec<KS> a;
  };
  struct B {
    float v[KS];
  };
  __device__ static __forceinline__ A load_a(const void* apack, int64_t T, int lane) {
    A r;
    r.a.load(static_cast<const float*>(apack) + (T * 64 + lane) * KS);
    return r;
  }
  __device__ static __forceinline__ B make_b(const RowSrc& src, int64_t i, bool ok, int g) {
    B b;
    const int64_t off = ok ? row_offset(src, i) : 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int t = 4 * s + g;
      b.v[s] = (ok && t < src.d) ? -2.0f * static_cast<float>(row_elem(src, off, t)) : 0.0f;
    }
    return b;
  }
  __device__ static __forceinline__ f4 mfma(const A& a, const B& b, f4 c) {
    f4 acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.v[0], b.v[0], c, 0, 0, 0);
#pragma unroll
    for (int s = 1; s < KS; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.a.v[s], b.v[s], acc, 0, 0, 0);
    return acc;
  }
};

// SplitOps (d <= 8): one v_mfma_f32_16x16x32_bf16 per tile.  Codewords and -2x are split into two
// bf16 terms (c = c1 + c2 + e_c, -2x = x1 + x2 + e_x, |e| <= 2^-16 |.|) and the four 8-element groups
// of the 32-long contraction hold c1.x1, c1.x2, c2.x1 and c2.x2: lane group g carries c1 (g < 2) or
// c2 (g >= 2) of codeword l % 16 and x1 (g even) or x2 (g odd) of row l % 16.  bf16 products are
// exact in fp32, so s is off by at most the split remainder 2^-15 sum_t |c_t| |2 x_t| plus the
// accumulation roundings; both enter the certification bound.  For bf16 rows and codebooks the split
// is exact (c2 = x2 = 0).
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct SplitOps {
  static constexpr int DM = 8;
  struct A {
    bf8 v;
  };
  struct B {
    bf8 v;
  };
  // codeword k of the packed book: 8 bf16 of c1, then 8 of c2 (32 bytes)
  __device__ static __forceinline__ A load_a(const void* apack, int64_t T, int lane) {
    A r;
    r.v = *reinterpret_cast<const bf8*>(static_cast<const uint16_t*>(apack) + (T * 16 + (lane & 15)) * 16 +
                                        (lane >> 5) * 8);
    return r;
  }
  __device__ static __forceinline__ B make_b(const RowSrc& src, int64_t i, bool ok, int g) {
    float v[8];
    if (src.type == ET_F64) {
      const int64_t off = ok ? row_offset(src, i) : 0;
#pragma unroll
      for (int t = 0; t < 8; ++t) v[t] = (ok && t < src.d) ? static_cast<float>(row_elem(src, off, t)) : 0.0f;
    } else {
      const int64_t off = ok ? row_offset(src, i) : 0;
      if (src.type == ET_F32)
        load_f32_elems<8>(static_cast<const float*>(src.base) + off, src.d, ok, v);
      else
        load_bf16_elems<8>(static_cast<const uint16_t*>(src.base) + off, src.d, ok, v);
    }
    return make_b_vals(v, g);
  }
  // the B operand of lane group g from the row's first 8 elements (zero past d)
  __device__ static __forceinline__ B make_b_vals(const float (&v)[8], int g) {
    u32x4 h;
#pragma unroll
    for (int q = 0; q < 4; ++q) h[q] = bf16x2_split(-2.0f * v[2 * q], -2.0f * v[2 * q + 1], (g & 1) != 0);
    B b;
    b.v = __builtin_bit_cast(bf8, h);
    return b;
  }
  __device__ static __forceinline__ f4 mfma(const A& a, const B& b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, c, 0, 0, 0);
  }
};

// Split-bf16 codebook pack: per codeword 8 bf16 of c1 then 8 of c2 (zero past d), and ||c||^2.
__global__ __launch_bounds__(256) void prep_codebook_split(const void* __restrict__ C, int ct, int64_t K, int d,
                                                           int64_t tiles, uint16_t* __restrict__ apack,
                                                           float* __restrict__ cnp, int* __restrict__ rcount) {
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (k == 0) *rcount = 0;
  if (k >= tiles * 16) return;
  float c[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) c[t] = (k < K && t < d) ? static_cast<float>(cb_elem(C, ct, k, d, t)) : 0.0f;
  float cn = 0.0f;
#pragma unroll
  for (int t = 0; t < 8; ++t) cn = cn + c[t] * c[t];
  cnp[k] = (k < K) ? cn : __builtin_inff();
  u16x8 hi, lo;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    uint16_t h, l;
    bf16_split(c[t], h, l);
    hi[t] = h;
    lo[t] = l;
  }
  u16x8* dst = reinterpret_cast<u16x8*>(apack + k * 16);
  dst[0] = hi;
  dst[1] = lo;
}

// ------------------------------------------------------------------------------------------------
// 2 + 3. MFMA screen with fused top-tile tracking, then exact re-scoring of the kept tiles
// ------------------------------------------------------------------------------------------------
template <class OPS, int NB, int CB, int NC>
__global__ __launch_bounds__(256) void screen_kernel(RowSrc src, const void* __restrict__ apack,
                                                     const float* __restrict__ cnp, int64_t tiles, int64_t tps,
                                                     const void* __restrict__ C, int ct, int64_t K,
                                                     int* __restrict__ pT, float* __restrict__ pM,
                                                     float* __restrict__ pR, double* __restrict__ pD,
                                                     int* __restrict__ pK, double* __restrict__ xn2o) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int jl = lane & 15;
  const int g = lane >> 4;
  const int split = blockIdx.y;
  const int64_t n = src.n;
  const int d = src.d;
  const int64_t row0 = (static_cast<int64_t>(blockIdx.x) * 4 + wave) * (16 * CB);
  if (row0 >= n) return;  // no barriers below: a wave past the end simply leaves

  typename OPS::B bop[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int64_t i = row0 + cb * 16 + jl;
    bop[cb] = OPS::make_b(src, i, i < n, g);
  }

  float m[CB][NB];
  int id[CB][NB];
  float rest[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    rest[cb] = __builtin_inff();
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      m[cb][j] = __builtin_inff();
      id[cb][j] = -1;
    }
  }

  const int64_t t0 = static_cast<int64_t>(split) * tps;
  const int64_t t1 = (t0 + tps < tiles) ? t0 + tps : tiles;
  if (t0 < t1) {
    // codebook tiles are loaded CRVQ_SCREEN_PREFETCH iterations ahead (clamped to the last tile)
    typename OPS::A a_q[CRVQ_SCREEN_PREFETCH];
    f4 c_q[CRVQ_SCREEN_PREFETCH];
#pragma unroll
    for (int u = 0; u < CRVQ_SCREEN_PREFETCH; ++u) {
      const int64_t Tu = (t0 + u < t1) ? t0 + u : t1 - 1;
      a_q[u] = OPS::load_a(apack, Tu, lane);
      c_q[u] = *reinterpret_cast<const f4*>(cnp + Tu * 16 + 4 * g);
    }
    // hands out tile T's operands and issues the load of tile T + CRVQ_SCREEN_PREFETCH
    auto advance = [&](int64_t T, typename OPS::A& a, f4& c4) {
      a = a_q[0];
      c4 = c_q[0];
#pragma unroll
      for (int u = 0; u + 1 < CRVQ_SCREEN_PREFETCH; ++u) {
        a_q[u] = a_q[u + 1];
        c_q[u] = c_q[u + 1];
      }
      const int64_t Tn = (T + CRVQ_SCREEN_PREFETCH < t1) ? T + CRVQ_SCREEN_PREFETCH : t1 - 1;
      a_q[CRVQ_SCREEN_PREFETCH - 1] = OPS::load_a(apack, Tn, lane);
      c_q[CRVQ_SCREEN_PREFETCH - 1] = *reinterpret_cast<const f4*>(cnp + Tn * 16 + 4 * g);
    };
    if constexpr (NB == 1) {
      // Top-1: tiles are taken in chunks of NC.  Inside a chunk every value only folds into the
      // chunk minimum (two v_min3 per tile and row); the kept-chunk and "rest" bookkeeping runs once
      // per chunk.  Full chunks run unguarded; a shorter last chunk tile by tile.
      float cm[CB];
      auto tile = [&](int64_t T) {
        typename OPS::A a;
        f4 c4;
        advance(T, a, c4);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
          const f4 acc = OPS::mfma(a, bop[cb], c4);
          cm[cb] = fminf(fminf(cm[cb], acc[0]), acc[1]);
          cm[cb] = fminf(fminf(cm[cb], acc[2]), acc[3]);
        }
      };
      auto fold = [&](int64_t T0) {
        const int Ci = static_cast<int>(T0);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
          rest[cb] = __builtin_amdgcn_fmed3f(m[cb][0], rest[cb], cm[cb]);
          const bool lt = cm[cb] < m[cb][0];
          m[cb][0] = fminf(m[cb][0], cm[cb]);
          id[cb][0] = lt ? Ci : id[cb][0];
          cm[cb] = __builtin_inff();
        }
      };
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) cm[cb] = __builtin_inff();
      int64_t T0 = t0;
      for (; T0 + NC <= t1; T0 += NC) {
#pragma unroll
        for (int u = 0; u < NC; ++u) tile(T0 + u);
        fold(T0);
      }
      if (T0 < t1) {
        for (int64_t T = T0; T < t1; ++T) tile(T);
        fold(T0);
      }
    } else {
      // Top-B: the minimum x of a tile (NC = 1) or of a chunk of NC tiles enters the sorted list of
      // the NB smallest, keyed by the first tile; what falls off the list joins "rest".
      auto insert = [&](int cb, float x, int Ti) {
          if constexpr (NB == 2) {
            // m0 <= m1 <= rest is kept sorted with medians: 10 VALU ops per tile and row
            const bool lt0 = x < m[cb][0];
            const bool lt1 = x < m[cb][1];
            rest[cb] = __builtin_amdgcn_fmed3f(m[cb][1], rest[cb], x);
            m[cb][1] = __builtin_amdgcn_fmed3f(m[cb][0], m[cb][1], x);
            m[cb][0] = fminf(m[cb][0], x);
            id[cb][1] = lt0 ? id[cb][0] : (lt1 ? Ti : id[cb][1]);
            id[cb][0] = lt0 ? Ti : id[cb][0];
          } else {
            int xi = Ti;
#pragma unroll
            for (int j = 0; j < NB; ++j) {
              const bool lt = x < m[cb][j];
              const float nv = fminf(x, m[cb][j]);
              const float cv = fmaxf(x, m[cb][j]);
              const int ni = lt ? xi : id[cb][j];
              xi = lt ? id[cb][j] : xi;
              m[cb][j] = nv;
              id[cb][j] = ni;
              x = cv;
            }
            rest[cb] = fminf(rest[cb], x);
          }
      };
      if constexpr (NC == 1) {
        for (int64_t T = t0; T < t1; ++T) {
          typename OPS::A a;
          f4 c4;
          advance(T, a, c4);
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) {
            const f4 acc = OPS::mfma(a, bop[cb], c4);
            insert(cb, fminf(fminf(acc[0], acc[1]), fminf(acc[2], acc[3])), static_cast<int>(T));
          }
        }
      } else {
        // long tile ranges: inside a chunk every value only folds into the chunk minimum, the list
        // insertion runs once per chunk
        for (int64_t T0 = t0; T0 < t1; T0 += NC) {
          const int64_t Te = (T0 + NC < t1) ? T0 + NC : t1;
          float xc[CB];
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) xc[cb] = __builtin_inff();
          for (int64_t T = T0; T < Te; ++T) {
            typename OPS::A a;
            f4 c4;
            advance(T, a, c4);
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) {
              const f4 acc = OPS::mfma(a, bop[cb], c4);
              xc[cb] = fminf(fminf(xc[cb], acc[0]), acc[1]);
              xc[cb] = fminf(fminf(xc[cb], acc[2]), acc[3]);
            }
          }
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) insert(cb, xc[cb], static_cast<int>(T0));
        }
      }
    }
  }

  if constexpr (NB == 1) {
    // Top-1.  The lane group whose kept chunk has the smallest minimum wins the row; the best chunks
    // of the other three groups join the bound ("rest").  The winner group's codewords of that chunk
    // (4 per tile) are re-scored exactly, lane group r taking codeword r of every tile, and reduced
    // in (D, k) order.  A row whose true minimum sits elsewhere fails certification later and is
    // re-searched exactly.
    constexpr int DM = OPS::DM;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int64_t i = row0 + cb * 16 + jl;
      const bool valid = i < n;
      const float mg = m[cb][0];
      float mw = mg;
      int gw = g;
#pragma unroll
      for (int msk = 16; msk <= 32; msk <<= 1) {
        const float om = __shfl_xor(mw, msk);
        const int og = __shfl_xor(gw, msk);
        const bool take = om < mw || (om == mw && og < gw);
        mw = take ? om : mw;
        gw = take ? og : gw;
      }
      float rr = (g == gw) ? rest[cb] : fminf(rest[cb], mg);
      rr = fminf(rr, __shfl_xor(rr, 16));
      rr = fminf(rr, __shfl_xor(rr, 32));
      const int Tw = __shfl(id[cb][0], jl + 16 * gw);
      double xd[DM];
      load_row_exact<DM>(src, i, valid, xd);
      double D = __builtin_inf();
      int kk = INT_MAX;
#pragma unroll
      for (int u0 = 0; u0 < NC; u0 += 4) {
        float cw[4][DM];
        bool ok[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int64_t T = static_cast<int64_t>(Tw) + u0 + u;
          const int64_t k = T * 16 + 4 * gw + g;
          ok[u] = valid && Tw >= 0 && u0 + u < NC && T < t1 && k < K;
          load_codeword<DM>(C, ct, k, d, ok[u], cw[u]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (ok[u]) {
            double Du = 0.0;
#pragma unroll
            for (int t = 0; t < DM; ++t) {
              if (t < d) {
                const double diff = xd[t] - static_cast<double>(cw[u][t]);
                Du = Du + diff * diff;
              }
            }
            const int ku = static_cast<int>((static_cast<int64_t>(Tw) + u0 + u) * 16 + 4 * gw + g);
            if (cless(Du, ku, D, kk)) {
              D = Du;
              kk = ku;
            }
          }
        }
      }
#pragma unroll
      for (int msk = 16; msk <= 32; msk <<= 1) {
        const double oD = __shfl_xor(D, msk);
        const int ok2 = __shfl_xor(kk, msk);
        const bool take = cless(oD, ok2, D, kk);
        D = take ? oD : D;
        kk = take ? ok2 : kk;
      }
      if (g == 0 && valid) {
        double xn2 = 0.0;
#pragma unroll
        for (int t = 0; t < DM; ++t)
          if (t < d) xn2 = xn2 + xd[t] * xd[t];
        pD[static_cast<int64_t>(split) * n + i] = D;
        pK[static_cast<int64_t>(split) * n + i] = kk;
        pR[static_cast<int64_t>(split) * n + i] = rr;
        if (split == 0) xn2o[i] = xn2;
      }
    }
  } else {
    // Top-B: per row and lane group the kept tile (or chunk) ids; per row the smallest minimum of
    // every other tile or chunk over the four lane groups (a lower bound on the screen value of every
    // codeword not kept).
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int64_t i = row0 + cb * 16 + jl;
      float rs = rest[cb];
      rs = fminf(rs, __shfl_xor(rs, 16));
      rs = fminf(rs, __shfl_xor(rs, 32));
      if (i < n) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          pT[((static_cast<int64_t>(split) * 4 + g) * NB + j) * n + i] = id[cb][j];
          pM[((static_cast<int64_t>(split) * 4 + g) * NB + j) * n + i] = m[cb][j];
        }
        if (g == 0) pR[static_cast<int64_t>(split) * n + i] = rs;
      }
    }
  }
}

// ------------------------------------------------------------------------------------------------
// 2'. top-1 screen on 32 x 32 tiles with split-fp16 operands (d <= 8, long codebooks)
// ------------------------------------------------------------------------------------------------
// Codewords and -2x are scaled by one power of two alpha (alpha max|c| in [2^11, 2^12)) and split
// into two fp16 terms: alpha c = c1 + c2 + e_c, alpha (-2x) = x1 + x2 + e_x with |e| <= 2^-22 |.|
// (plus 2^-25 below the fp16 normal range).  Per 32 x 32 tile two v_mfma_f32_32x32x16_f16 form
//   alpha^2 s = c1.x1 + c2.x1  (first: lanes 0-31 carry c1 / x1, lanes 32-63 c2 / x1)
//             + c1.x2 + N      (second: lanes 0-31 c1 / x2, lanes 32-63 the three fp16 terms of
//                               N 2^-12, N = sum_t (alpha c_t)^2, against 2^12)
// fp16 products are exact in fp32.  The dropped c2.x2, the split remainders and the accumulation
// roundings enter the certification bound.  Lane l ends with the 16 values of codewords
// 8 (r / 4) + 4 (l / 32) + r % 4, r = 0..15, for row l % 32.  A row with an element whose scaled
// value does not fit fp16 is not screened: its bound is set to -inf, so it is re-searched exactly.
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));

constexpr int kS32Tile = 32;         // codewords per tile
constexpr int64_t kRescueBlocks = 1024;  // persistent grid of the exact rescue
constexpr int kRescueParts = 16;         // codeword ranges of a parted top-1 rescue
constexpr int64_t kRescuePartMinK = 8192;  // codebooks from which the top-1 rescue is parted
constexpr int64_t kS32SharedRowsMaxN = int64_t{1} << 23;  // second screen: shared rows below this n
constexpr int kS32TileHalves = 768;  // packed fp16 per tile: c1, c2, N terms, 32 x 8 each
constexpr int kS32MaxParts = 256;    // partial maxima of the codebook scale reduction

// ------------------------------------------------------------------------------------------------
// Certified tile skipping for the long top-1 screen.  For any codeword c and row x,
//   | ||x|| - ||c|| | <= ||x - c||   and   | x_t - c_t | <= ||x - c||   (any coordinate t),
// so once a row's best distance is known to be at most D_up, a codeword whose norm, coordinate j or
// coordinate q lies further than sqrt(D_up) from the row's can neither win nor tie.  Codewords are
// packed in the order of a key (norm bin major, then the bin of coordinate j, then the bin of
// coordinate q), rows are screened in the order of the same key, and each wave keeps, per pair of
// tiles ("chunk" of 64 codewords), the ranges of the codewords' norms and coordinates j and q: a
// chunk outside every row's band in any of the three is skipped.  D_up comes from
// the wave's running screen minimum m:  D(c_m) <= m / alpha^2 + ||x||^2 + delta, delta the screen's
// error bound taken with R = the largest codeword norm.  Every quantity is in units of the codebook
// scale alpha (exact powers of two), rounded outward, so the test is conservative; a skipped
// codeword is strictly worse than the kept chunk's exact winner, so the certificate and the results
// are those of the full screen.
constexpr int kPruneBins1 = 16;                // norm bins (major key)
constexpr int kPruneBins2 = 16;                // bins of coordinate j (middle key)
constexpr int kPruneBins3 = 64;                // bins of coordinate q (minor key)
constexpr int kPruneKeys = kPruneBins1 * kPruneBins2 * kPruneBins3;
constexpr int kPruneFine = 4096;               // fine bins of each key feature (quantile edges)
constexpr int64_t kPruneMinRows = 32768;       // rows from which the screen is pruned

struct PruneData {
  const int* corder;        // sorted codeword position -> codeword
  const int* coff;          // first sorted position of every key
  const uint4* cbnd;        // per chunk: ordered keys of {min, max} scaled norm, {min, max} scaled c_j
  const uint2* cbnd3;       // per chunk: ordered keys of {min, max} scaled c_q
  const uint32_t* cminS;    // suffix minimum over chunks of the norm minimum key
  const uint32_t* cmaxP;    // prefix maximum over chunks of the norm maximum key
  const int* rord;          // rows in key order
  const int* rkey;          // key of every row
  const float* prm;         // {max ||c||, min c_j, max c_j, scaled max ||c|| rounded up, min c_q, max c_q}
  const float* lD;          // second screen: per listed row, its first-screen exact distance rounded up
  int jp;                   // the coordinate j
  int jq;                   // the coordinate q
};

// Order-preserving map of a float (both zeros to the same key) to an unsigned integer, so that wave
// uniform comparisons run on the scalar unit.
__device__ __forceinline__ uint32_t okey(float f) {
  const uint32_t u = (f == 0.0f) ? 0u : __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float okey_inv(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}
// float just below / above a non-negative double
__device__ __forceinline__ float f32_down(double x) {
  float f = static_cast<float>(x);
  if (static_cast<double>(f) > x) f = (f > 0.0f) ? __uint_as_float(__float_as_uint(f) - 1u) : -__uint_as_float(1u);
  return f;
}
__device__ __forceinline__ float f32_up(double x) {
  float f = static_cast<float>(x);
  if (static_cast<double>(f) < x) f = (f >= 0.0f) ? __uint_as_float(__float_as_uint(f) + 1u) : -0.0f;
  return f;
}

// The float next to finite f towards +inf / -inf (bit steps; a zero steps to the smallest subnormal).
__device__ __forceinline__ float f32_next_up(float f) {
  if (f == 0.0f) return __uint_as_float(1u);
  const uint32_t u = __float_as_uint(f);
  return __uint_as_float(f > 0.0f ? u + 1u : u - 1u);
}
__device__ __forceinline__ float f32_next_down(float f) { return -f32_next_up(-f); }
// float at or below / at or above any double (the bounds of a band that may be negative)
__device__ __forceinline__ float f32_down_any(double x) {
  float f = static_cast<float>(x);
  if (static_cast<double>(f) > x) f = f32_next_down(f);
  return f;
}
__device__ __forceinline__ float f32_up_any(double x) {
  float f = static_cast<float>(x);
  if (static_cast<double>(f) < x) f = f32_next_up(f);
  return f;
}

// Bin of x in [lo, hi] out of nb (clamped; one bin when the range is empty).
__device__ __forceinline__ int prune_bin(float x, float lo, float hi, int nb) {
  const float span = hi - lo;
  float f = (span > 0.0f) ? (x - lo) * (static_cast<float>(nb) / span) : 0.0f;
  f = fminf(fmaxf(f, 0.0f), static_cast<float>(nb - 1));
  return static_cast<int>(f);
}

// Fine bin of feature value x over [lo, hi] (clamped).
__device__ __forceinline__ int prune_fine(float x, float lo, float hi) { return prune_bin(x, lo, hi, kPruneFine); }

// The three key features of a vector: ||v||, v_j, v_q.
__device__ __forceinline__ void prune_features(const float (&v)[8], int jp, int jq, float (&f)[3]) {
  float n2 = 0.0f, xj = 0.0f, xq = 0.0f;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    n2 = n2 + v[t] * v[t];
    xj = (t == jp) ? v[t] : xj;
    xq = (t == jq) ? v[t] : xq;
  }
  f[0] = sqrtf(n2);
  f[1] = xj;
  f[2] = xq;
}

// Fine bins of the features, r = {max ||c||, min c_j, max c_j, min c_q, max c_q}.
__device__ __forceinline__ void prune_fine3(const float (&f)[3], const float (&r)[5], int (&b)[3]) {
  b[0] = prune_fine(f[0], 0.0f, fmaxf(r[0], 0x1p-126f));
  b[1] = prune_fine(f[1], r[1], r[2]);
  b[2] = prune_fine(f[2], r[3], r[4]);
}

constexpr int kPruneTile = 4096;  // codewords per block of the fine histograms
// threads and vectors per block of the key counting and scatter, codebook and rows
#ifndef CRVQ_PRUNE_CB_NT
#define CRVQ_PRUNE_CB_NT 1024
#endif
#ifndef CRVQ_PRUNE_CB_TILE
#define CRVQ_PRUNE_CB_TILE 4096
#endif
#ifndef CRVQ_PRUNE_ROW_NT
#define CRVQ_PRUNE_ROW_NT 1024
#endif
#ifndef CRVQ_PRUNE_ROW_TILE
#define CRVQ_PRUNE_ROW_TILE 8192
#endif
constexpr int kPruneCbThreads = CRVQ_PRUNE_CB_NT, kPruneCbTile = CRVQ_PRUNE_CB_TILE;
constexpr int kPruneRowThreads = CRVQ_PRUNE_ROW_NT, kPruneRowTile = CRVQ_PRUNE_ROW_TILE;
constexpr int kPruneParts = 256;  // partial blocks of the binning ranges

// Partial ranges of the codebook's key features (max norm, min and max of coordinates j and q) over a
// strided share of the codewords, and (every block a share) the cleared key counts of codewords and
// rows and the cleared fine histograms.
__global__ __launch_bounds__(256) void prune_stats_partial(const void* __restrict__ C, int ct, int64_t K, int d,
                                                           int jp, int jq, float* __restrict__ part,
                                                           int* __restrict__ hist2) {
  __shared__ float s_r[5][256];
  const int tid = threadIdx.x;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + tid; e < 2 * kPruneKeys + 3 * kPruneFine; e += gridDim.x * 256)
    hist2[e] = 0;
  float r[5] = {0.0f, __builtin_inff(), -__builtin_inff(), __builtin_inff(), -__builtin_inff()};
  for (int64_t k = static_cast<int64_t>(blockIdx.x) * 256 + tid; k < K; k += static_cast<int64_t>(gridDim.x) * 256) {
    float v[8];
    if (ct == ET_F32)
      load_f32_elems<8>(static_cast<const float*>(C) + k * d, d, true, v);
    else
      load_bf16_elems<8>(static_cast<const uint16_t*>(C) + k * d, d, true, v);
    float n2 = 0.0f, cj = 0.0f, cq = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      n2 = n2 + v[t] * v[t];
      cj = (t == jp) ? v[t] : cj;
      cq = (t == jq) ? v[t] : cq;
    }
    r[0] = fmaxf(r[0], sqrtf(n2));
    r[1] = fminf(r[1], cj);
    r[2] = fmaxf(r[2], cj);
    r[3] = fminf(r[3], cq);
    r[4] = fmaxf(r[4], cq);
  }
#pragma unroll
  for (int q = 0; q < 5; ++q) s_r[q][tid] = r[q];
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (tid < w) {
      s_r[0][tid] = fmaxf(s_r[0][tid], s_r[0][tid + w]);
      s_r[1][tid] = fminf(s_r[1][tid], s_r[1][tid + w]);
      s_r[2][tid] = fmaxf(s_r[2][tid], s_r[2][tid + w]);
      s_r[3][tid] = fminf(s_r[3][tid], s_r[3][tid + w]);
      s_r[4][tid] = fmaxf(s_r[4][tid], s_r[4][tid + w]);
    }
    __syncthreads();
  }
  if (tid == 0) {
#pragma unroll
    for (int q = 0; q < 5; ++q) part[q * kPruneParts + blockIdx.x] = s_r[q][0];
  }
}

// Every block folds the partial ranges r = {max ||c||, min c_j, max c_j, min c_q, max c_q} (the
// first one also publishes them to prm[0..2] and prm[4..5]).
__device__ __forceinline__ void prune_fold_ranges(const float* __restrict__ part, int nparts, float* __restrict__ prm,
                                                  float (&r)[5]) {
  // (blocks of 256 threads or more; the first 256 fold the 256 partial ranges)
  static_assert(kPruneParts == 256, "the fold halves 256 entries");
  __shared__ float s_r[5][kPruneParts];
  const int tid = threadIdx.x;
  if (tid < kPruneParts) {
    const bool in = tid < nparts;
    s_r[0][tid] = in ? part[tid] : 0.0f;
    s_r[1][tid] = in ? part[kPruneParts + tid] : __builtin_inff();
    s_r[2][tid] = in ? part[2 * kPruneParts + tid] : -__builtin_inff();
    s_r[3][tid] = in ? part[3 * kPruneParts + tid] : __builtin_inff();
    s_r[4][tid] = in ? part[4 * kPruneParts + tid] : -__builtin_inff();
  }
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (tid < w) {
      s_r[0][tid] = fmaxf(s_r[0][tid], s_r[0][tid + w]);
      s_r[1][tid] = fminf(s_r[1][tid], s_r[1][tid + w]);
      s_r[2][tid] = fmaxf(s_r[2][tid], s_r[2][tid + w]);
      s_r[3][tid] = fminf(s_r[3][tid], s_r[3][tid + w]);
      s_r[4][tid] = fmaxf(s_r[4][tid], s_r[4][tid + w]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int q = 0; q < 5; ++q) r[q] = s_r[q][0];
  if (blockIdx.x == 0 && tid == 0) {
    prm[0] = r[0];
    prm[1] = r[1];
    prm[2] = r[2];
    prm[4] = r[3];
    prm[5] = r[4];
  }
}

// The key features of vector i of src (the rows, or the codewords as a set of K rows).
__device__ __forceinline__ void prune_vec_features(const RowSrc& src, int64_t i, int jp, int jq, float (&f)[3]) {
  float v[8];
  const int64_t off = row_offset(src, i);
  if (src.type == ET_F32) {
    load_f32_elems<8>(static_cast<const float*>(src.base) + off, src.d, true, v);
  } else if (src.type == ET_BF16) {
    load_bf16_elems<8>(static_cast<const uint16_t*>(src.base) + off, src.d, true, v);
  } else {  // fp64 rows (residuals), rounded to fp32 as the screen's operands are: the key only orders
#pragma unroll
    for (int t = 0; t < 8; ++t) v[t] = t < src.d ? static_cast<float>(static_cast<const double*>(src.base)[off + t]) : 0.0f;
  }
  prune_features(v, jp, jq, f);
}

// Fine histograms of the codebook's three key features over their ranges (kPruneTile codewords per
// block of NT threads, counted in LDS, nonzero counts added to fine[3][kPruneFine] with integer atomics).
template <int NT>
__global__ __launch_bounds__(NT) void prune_fine_kernel(RowSrc cbs, int jp, int jq, const float* __restrict__ part,
                                                        int nparts, float* __restrict__ prm, int* __restrict__ fine) {
  static_assert(kPruneTile % NT == 0, "whole rounds");
  __shared__ int h[3 * kPruneFine];
  float r[5];
  prune_fold_ranges(part, nparts, prm, r);
  const int tid = threadIdx.x;
  for (int b = tid; b < 3 * kPruneFine; b += NT) h[b] = 0;
  __syncthreads();
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * kPruneTile;
  for (int q = 0; q < kPruneTile / NT; ++q) {
    const int64_t i = i0 + q * NT + tid;
    if (i < cbs.n) {
      float f[3];
      int b[3];
      prune_vec_features(cbs, i, jp, jq, f);
      prune_fine3(f, r, b);
#pragma unroll
      for (int a = 0; a < 3; ++a) atomicAdd(h + a * kPruneFine + b[a], 1);
    }
  }
  __syncthreads();
  for (int b = tid; b < 3 * kPruneFine; b += NT)
    if (h[b]) atomicAdd(fine + b, h[b]);
}

// Coarse bin of every fine bin from the codebook's fine histograms: nb equal-width bins over a
// robust range of the feature, median +- 3 interquartile ranges (about +-4 sigma for normal data, the
// whole range of the codewords there), with the values outside it in the end bins, so that heavy
// tails and outlier columns do not squeeze the bulk of the codewords into one bin.  256 threads,
// 16 fine bins each.
__device__ __forceinline__ void prune_build_lut(const int* __restrict__ fine, uint8_t (*lut)[kPruneFine],
                                                int* scan) {
  __shared__ int s_q[3];
  const int tid = threadIdx.x;
  constexpr int kPer = kPruneFine / 256;
  const int nb[3] = {kPruneBins1, kPruneBins2, kPruneBins3};
  for (int a = 0; a < 3; ++a) {
    int c[kPer];
    int sum = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      c[q] = fine[a * kPruneFine + tid * kPer + q];
      sum += c[q];
    }
    scan[tid] = sum;
    if (tid < 3) s_q[tid] = 0;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {
      const int v = tid >= o ? scan[tid - o] : 0;
      __syncthreads();
      scan[tid] += v;
      __syncthreads();
    }
    const int64_t total = scan[255];
    // the fine bins holding the quartiles: quartile u is the first bin whose cumulative count exceeds
    // u * total / 4 (exactly one thread owns it)
    {
      int64_t run = scan[tid] - sum;
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int64_t nxt = run + c[q];
#pragma unroll
        for (int u = 0; u < 3; ++u) {
          const int64_t tgt = (total * (u + 1)) / 4;
          if (run <= tgt && tgt < nxt) s_q[u] = tid * kPer + q;
        }
        run = nxt;
      }
    }
    __syncthreads();
    const int iqr = s_q[2] - s_q[0];
    int flo = s_q[1] - 3 * iqr - 1, fhi = s_q[1] + 3 * iqr + 1;
    flo = flo < 0 ? 0 : flo;
    fhi = fhi > kPruneFine - 1 ? kPruneFine - 1 : fhi;
    const int span = fhi - flo + 1;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int f = tid * kPer + q;
      int cb = f < flo ? 0 : ((f - flo) * nb[a]) / span;
      cb = cb < nb[a] ? cb : nb[a] - 1;
      lut[a][f] = static_cast<uint8_t>(cb);
    }
    __syncthreads();
  }
}

// The lookup table of prune_build_lut, built once (one block) into lut_g[3][kPruneFine].
__global__ __launch_bounds__(256) void prune_lut_kernel(const int* __restrict__ fine, uint8_t* __restrict__ lut_g) {
  __shared__ uint8_t lut[3][kPruneFine];
  __shared__ int scan[256];
  prune_build_lut(fine, lut, scan);
  const uint4* src = reinterpret_cast<const uint4*>(&lut[0][0]);
  uint4* dst = reinterpret_cast<uint4*>(lut_g);
  for (int e = threadIdx.x; e < 3 * kPruneFine / 16; e += 256) dst[e] = src[e];
}

// Keys of TILE vectors per block of NT threads, counted in LDS, the block's nonzero counts added to
// the global counts (one integer atomic per key present in the block).  The LDS counters cost the
// same per block whatever its tile, so larger tiles and blocks spread them over more vectors.
template <int NT, int TILE>
__global__ __launch_bounds__(NT) void prune_count_kernel(RowSrc src, int jp, int jq, const float* __restrict__ part,
                                                         int nparts, float* __restrict__ prm,
                                                         const uint8_t* __restrict__ lut_g, int* __restrict__ keys,
                                                         int* __restrict__ hist) {
  static_assert(TILE % NT == 0 && kPruneKeys % (4 * NT) == 0, "whole rounds");
  __shared__ int h[kPruneKeys];
  __shared__ uint8_t lut[3][kPruneFine];
  float r[5];
  prune_fold_ranges(part, nparts, prm, r);
  const int tid = threadIdx.x;
  for (int e = tid; e < 3 * kPruneFine / 16; e += NT)
    reinterpret_cast<uint4*>(&lut[0][0])[e] = reinterpret_cast<const uint4*>(lut_g)[e];
  for (int b = tid; b < kPruneKeys / 4; b += NT) reinterpret_cast<int4*>(h)[b] = make_int4(0, 0, 0, 0);
  __syncthreads();
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * TILE;
  for (int q = 0; q < TILE / NT; ++q) {
    const int64_t i = i0 + q * NT + tid;
    if (i < src.n) {
      float f[3];
      int b[3];
      prune_vec_features(src, i, jp, jq, f);
      prune_fine3(f, r, b);
      const int key = (static_cast<int>(lut[0][b[0]]) * kPruneBins2 + lut[1][b[1]]) * kPruneBins3 + lut[2][b[2]];
      keys[i] = key;
      atomicAdd(h + key, 1);
    }
  }
  __syncthreads();
  for (int b = tid; b < kPruneKeys; b += NT)
    if (h[b]) atomicAdd(hist + b, h[b]);
}

// Exclusive prefix sums of the key counts, in place (the scatter's cursors), and a copy in off.
__global__ __launch_bounds__(1024) void prune_scan_kernel(int* __restrict__ hist, int* __restrict__ off) {
  __shared__ int sh[1024];
  constexpr int kPer = kPruneKeys / 1024;
  const int t = threadIdx.x;
  int v[kPer];
  int sum = 0;
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    v[q] = hist[t * kPer + q];
    sum += v[q];
  }
  sh[t] = sum;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const int a = t >= o ? sh[t - o] : 0;
    __syncthreads();
    sh[t] += a;
    __syncthreads();
  }
  int run = t > 0 ? sh[t - 1] : 0;
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    hist[t * kPer + q] = run;
    if (off) off[t * kPer + q] = run;
    run += v[q];
  }
}

// order[...] = i in key order: ranks within the block from LDS counters, one global cursor advance
// per key present in the block.  The order within a key is not fixed; results do not depend on it.
template <int NT, int TILE>
__global__ __launch_bounds__(NT) void prune_order_kernel(const int* __restrict__ keys, int64_t n,
                                                         int* __restrict__ cursor, int* __restrict__ order) {
  static_assert(TILE % NT == 0 && kPruneKeys % (4 * NT) == 0, "whole rounds");
  __shared__ int h[kPruneKeys];
  const int tid = threadIdx.x;
  for (int b = tid; b < kPruneKeys / 4; b += NT) reinterpret_cast<int4*>(h)[b] = make_int4(0, 0, 0, 0);
  __syncthreads();
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * TILE;
  constexpr int kQ = TILE / NT;
  int key[kQ], rank[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    const int64_t i = i0 + q * NT + tid;
    key[q] = i < n ? keys[i] : -1;
    rank[q] = key[q] >= 0 ? atomicAdd(h + key[q], 1) : 0;
  }
  __syncthreads();
  for (int b = tid; b < kPruneKeys; b += NT)
    if (h[b]) h[b] = atomicAdd(cursor + b, h[b]);
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    const int64_t i = i0 + q * NT + tid;
    if (key[q] >= 0) {
      const int pos = h[key[q]] + rank[q];
      if (pos >= 0 && pos < n) order[pos] = static_cast<int>(i);
    }
  }
}

__global__ __launch_bounds__(256) void prune_fill_kernel(int* __restrict__ p, int64_t n, int v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

// Per chunk (sorted positions 64 c .. 64 c + 63, one wave): the range of alpha ||c|| (fp64, rounded
// outward) and of alpha c_j and alpha c_q (exact), as ordered keys; an empty chunk gets empty ranges.
__global__ __launch_bounds__(256) void prune_chunks_kernel(const void* __restrict__ C, int ct, int64_t K, int d, int jp,
                                                           int jq, const int* __restrict__ corder,
                                                           const float* __restrict__ alpha_p, int64_t nch,
                                                           uint4* __restrict__ cbnd, uint2* __restrict__ cbnd3) {
  const int lane = threadIdx.x & 63;
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (c >= nch) return;  // whole waves
  const double a = static_cast<double>(alpha_p[0]);
  double lo1 = __builtin_inf(), hi1 = -__builtin_inf();
  float lo2 = __builtin_inff(), hi2 = -__builtin_inff(), lo3 = __builtin_inff(), hi3 = -__builtin_inff();
  const int64_t q = 64 * c + lane;
  const int64_t k = q < K ? corder[q] : -1;
  if (k >= 0 && k < K) {
    float v[8];
    if (ct == ET_F32)
      load_f32_elems<8>(static_cast<const float*>(C) + k * d, d, true, v);
    else
      load_bf16_elems<8>(static_cast<const uint16_t*>(C) + k * d, d, true, v);
    double n2 = 0.0;
    float cj = 0.0f, cq = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      n2 = n2 + static_cast<double>(v[t]) * static_cast<double>(v[t]);
      cj = (t == jp) ? v[t] : cj;
      cq = (t == jq) ? v[t] : cq;
    }
    lo1 = hi1 = sqrt(n2) * a;
    lo2 = hi2 = cj * static_cast<float>(a);  // exact: a power of two, alpha |c| < 2^12
    lo3 = hi3 = cq * static_cast<float>(a);
  }
#pragma unroll
  for (int sh = 1; sh < 64; sh <<= 1) {
    const double o1 = __shfl_xor(lo1, sh), o2 = __shfl_xor(hi1, sh);
    lo1 = o1 < lo1 ? o1 : lo1;
    hi1 = o2 > hi1 ? o2 : hi1;
    lo2 = fminf(lo2, __shfl_xor(lo2, sh));
    hi2 = fmaxf(hi2, __shfl_xor(hi2, sh));
    lo3 = fminf(lo3, __shfl_xor(lo3, sh));
    hi3 = fmaxf(hi3, __shfl_xor(hi3, sh));
  }
  if (lane == 0) {
    uint4 b;
    b.x = okey(lo1 <= hi1 ? f32_down(lo1) : __builtin_inff());
    b.y = okey(lo1 <= hi1 ? f32_up(hi1) : -__builtin_inff());
    b.z = okey(lo2);
    b.w = okey(hi2);
    cbnd[c] = b;
    cbnd3[c] = make_uint2(okey(lo3), okey(hi3));
  }
}

// Envelopes for the wave's stop tests (suffix minimum of the norm minima, prefix maximum of the
// norm maxima) and the largest scaled codeword norm (rounded up) for the screen bound.
__global__ __launch_bounds__(1024) void prune_envelope_kernel(const uint4* __restrict__ cbnd, int nch,
                                                              uint32_t* __restrict__ cminS, uint32_t* __restrict__ cmaxP,
                                                              float* __restrict__ prm) {
  __shared__ uint32_t smin[1024], smax[1024];
  const int t = threadIdx.x;
  const uint4 b = t < nch ? cbnd[t] : make_uint4(0xffffffffu, 0u, 0u, 0u);
  smin[t] = b.x;  // suffix min: scan from the end
  smax[t] = b.y;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const uint32_t a = (t + o < 1024) ? smin[t + o] : 0xffffffffu;
    const uint32_t c = (t >= o) ? smax[t - o] : 0u;
    __syncthreads();
    smin[t] = smin[t] < a ? smin[t] : a;
    smax[t] = smax[t] > c ? smax[t] : c;
    __syncthreads();
  }
  if (t < nch) {
    cminS[t] = smin[t];
    cmaxP[t] = smax[t];
  }
  if (t == 0) prm[3] = fmaxf(okey_inv(smax[nch - 1]), 0.0f);
}

// The wave's walk over the chunks: two lists in LDS, the chunks above the start in ascending order
// (U) and those below it in descending order (D), consumed alternately (U[ui], D[di], ...).  After
// each narrowing of the bands the unvisited rest of each list is filtered in place, one chunk per
// lane: a chunk leaves it when outside a band, and a list ends at the first chunk past its side's
// envelope (every later chunk of that side is outside too).  The positions, lengths and bands are
// wave-uniform scalars; taking a chunk is one LDS read.
struct PruneCursor {
  int ui, un, di, dn, turn;
  uint32_t lo1, hi1, lo2, hi2, lo3, hi3;
};

__device__ __forceinline__ uint32_t rfl(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ bool prune_keep(const uint4& b, const uint2& b3, const PruneCursor& s) {
  return !((b.y < s.lo1) | (b.x > s.hi1) | (b.w < s.lo2) | (b.z > s.hi2) | (b3.y < s.lo3) | (b3.x > s.hi3));
}

// L[i0 .. n) filtered under the current bands into L[0 ..); returns the new length.  Four groups of
// 64 entries are examined per round, all their loads issued before any is used.
__device__ __forceinline__ int prune_filter(uint16_t* L, int i0, int n, bool up, const PruneCursor& s,
                                            const PruneData& pd, int lane) {
  constexpr int kG = 4;
  int w = 0;
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
  for (int b = i0; b < n; b += 64 * kG) {
    int c[kG];
    uint32_t env[kG];
    uint4 bd[kG];
    uint2 bd3[kG];
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      const int i = b + 64 * g + lane;
      c[g] = i < n ? static_cast<int>(L[i]) : -1;
    }
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      const int cc = c[g] >= 0 ? c[g] : 0;
      env[g] = up ? pd.cminS[cc] : pd.cmaxP[cc];
      bd[g] = pd.cbnd[cc];
      bd3[g] = pd.cbnd3[cc];
    }
    bool stop = false;
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      const bool valid = c[g] >= 0;
      const bool end = !valid || (up ? (env[g] > s.hi1) : (env[g] < s.lo1));
      const bool keep = !end & prune_keep(bd[g], bd3[g], s);
      const uint64_t em = __ballot(end);
      uint64_t km = __ballot(keep);
      if (em) km &= (uint64_t{1} << __builtin_ctzll(em)) - 1ull;  // nothing from the first end on
      if (!stop) {
        if ((km >> lane) & 1ull) L[w + __popcll(km & lt)] = static_cast<uint16_t>(c[g]);
        w += __popcll(km);
      }
      stop = stop || em != 0ull;
    }
    if (stop) break;
  }
  return static_cast<int>(rfl(static_cast<uint32_t>(w)));
}

// The next chunk to screen, or -1 when both lists are exhausted.
__device__ __forceinline__ int prune_take(PruneCursor& s, const uint16_t* U, const uint16_t* D) {
  if (s.ui < s.un && (s.turn == 0 || s.di >= s.dn)) {
    s.turn = 1;
    return static_cast<int>(rfl(U[s.ui++]));
  }
  if (s.di < s.dn) {
    s.turn = 0;
    return static_cast<int>(rfl(D[s.di++]));
  }
  return -1;
}

// New bands from the rows' running minima m (each lane: the rows of its column blocks, both lane
// halves of a row hold its two halves of every tile); band terms of row (cb, j) at sb[cb * 128 + k * 32 + j].
template <int CB>
__device__ __forceinline__ void prune_band(PruneCursor& s, const float (&m)[CB], const float* sb, int j) {
  float lo1 = __builtin_inff(), hi1 = -__builtin_inff(), lo2 = __builtin_inff(), hi2 = -__builtin_inff();
  float lo3 = __builtin_inff(), hi3 = -__builtin_inff();
  bool open = false;
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const float mr = fminf(m[cb], __shfl_xor(m[cb], 32));
    const float A = sb[cb * 128 + j], P = sb[cb * 128 + 32 + j], Q = sb[cb * 128 + 64 + j], B = sb[cb * 128 + 96 + j];
    if (B >= 0.0f) {
      if (!(mr < __builtin_inff())) {
        open = true;
      } else {
        // every operation below errs by at most 2^-24 of its operands; the margins are 16x that
        const float Dup = fmaxf((mr + B) + 0x1p-20f * (fabsf(mr) + B) + 0x1p-10f, 0.0f);
        const float r = sqrtf(Dup) * (1.0f + 0x1p-20f);
        const float s1 = 0x1p-20f * (A + r) + 0x1p-10f, s2 = 0x1p-20f * (fabsf(P) + r) + 0x1p-10f;
        const float s3 = 0x1p-20f * (fabsf(Q) + r) + 0x1p-10f;
        lo1 = fminf(lo1, (A - r) - s1);
        hi1 = fmaxf(hi1, (A + r) + s1);
        lo2 = fminf(lo2, (P - r) - s2);
        hi2 = fmaxf(hi2, (P + r) + s2);
        lo3 = fminf(lo3, (Q - r) - s3);
        hi3 = fmaxf(hi3, (Q + r) + s3);
      }
    }
  }
  if (open) {
    lo1 = lo2 = lo3 = -__builtin_inff();
    hi1 = hi2 = hi3 = __builtin_inff();
  }
#pragma unroll
  for (int sh = 1; sh < 64; sh <<= 1) {
    lo1 = fminf(lo1, __shfl_xor(lo1, sh));
    hi1 = fmaxf(hi1, __shfl_xor(hi1, sh));
    lo2 = fminf(lo2, __shfl_xor(lo2, sh));
    hi2 = fmaxf(hi2, __shfl_xor(hi2, sh));
    lo3 = fminf(lo3, __shfl_xor(lo3, sh));
    hi3 = fmaxf(hi3, __shfl_xor(hi3, sh));
  }
  s.lo1 = rfl(okey(lo1));
  s.hi1 = rfl(okey(hi1));
  s.lo2 = rfl(okey(lo2));
  s.hi2 = rfl(okey(hi2));
  s.lo3 = rfl(okey(lo3));
  s.hi3 = rfl(okey(hi3));
}

// min(c, a[0..15]) as a depth-3 tree of eight v_min3
__device__ __forceinline__ float min_fold16(float c, const f16v& a) {
  const float m0 = fminf(fminf(a[0], a[1]), a[2]);
  const float m1 = fminf(fminf(a[3], a[4]), a[5]);
  const float m2 = fminf(fminf(a[6], a[7]), a[8]);
  const float m3 = fminf(fminf(a[9], a[10]), a[11]);
  const float m4 = fminf(fminf(a[12], a[13]), a[14]);
  const float n0 = fminf(fminf(m0, m1), m2);
  const float n1 = fminf(fminf(m3, m4), a[15]);
  return fminf(fminf(c, n0), n1);
}

__device__ __forceinline__ uint16_t f16_bits(float v) { return __builtin_bit_cast(uint16_t, static_cast<_Float16>(v)); }
__device__ __forceinline__ float f16_val(uint16_t b) { return static_cast<float>(__builtin_bit_cast(_Float16, b)); }

// Partial maxima of |c| over the codebook (block b covers a strided share).
__global__ __launch_bounds__(256) void cb_absmax_partial(const void* __restrict__ C, int ct, int64_t count,
                                                         float* __restrict__ part) {
  __shared__ float sh[256];
  float m = 0.0f;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; e < count;
       e += static_cast<int64_t>(gridDim.x) * 256) {
    const float v = (ct == ET_F32) ? static_cast<const float*>(C)[e]
                                   : bf16_to_f(static_cast<const uint16_t*>(C)[e]);
    m = fmaxf(m, fabsf(v));
  }
  sh[threadIdx.x] = m;
  __syncthreads();
  for (int s = 128; s >= 1; s >>= 1) {
    if (static_cast<int>(threadIdx.x) < s) sh[threadIdx.x] = fmaxf(sh[threadIdx.x], sh[threadIdx.x + s]);
    __syncthreads();
  }
  if (threadIdx.x == 0) part[blockIdx.x] = sh[0];
}

// alpha = 2^(11 - floor(log2 max)), at most 2^126; 1 for an all-zero or non-finite codebook.
__device__ __forceinline__ float s32_alpha(float mx) {
  if (!(mx > 0.0f) || !(mx <= 3.402823466e38f)) return 1.0f;
  int e = ilogbf(mx);
  int s = 11 - e;
  if (s > 126) s = 126;
  return ldexpf(1.0f, s);
}

// Every block folds the partial maxima, block 0 publishes alpha; then thread k packs codeword k.
__global__ __launch_bounds__(256) void prep_codebook_s32(const void* __restrict__ C, int ct, int64_t K, int d,
                                                         int64_t tiles, const float* __restrict__ part, int nparts,
                                                         const int* __restrict__ corder,
                                                         uint16_t* __restrict__ apack, float* __restrict__ alpha_out,
                                                         int* __restrict__ rcount) {
  __shared__ float sh[256];
  sh[threadIdx.x] = (static_cast<int>(threadIdx.x) < nparts) ? part[threadIdx.x] : 0.0f;
  __syncthreads();
  for (int s = 128; s >= 1; s >>= 1) {
    if (static_cast<int>(threadIdx.x) < s) sh[threadIdx.x] = fmaxf(sh[threadIdx.x], sh[threadIdx.x + s]);
    __syncthreads();
  }
  const float alpha = s32_alpha(sh[0]);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    alpha_out[0] = alpha;
    rcount[0] = 0;  // rows left uncertain by the first screen
    rcount[1] = 0;  // rows left uncertain by the second (split) screen of those
  }
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (k >= tiles * kS32Tile) return;
  // position k holds codeword corder[k] when the book is packed in key order
  int64_t ks = (k < K) ? (corder ? static_cast<int64_t>(corder[k]) : k) : -1;
  if (ks >= K) ks = -1;
  float c[8];
#pragma unroll
  for (int t = 0; t < 8; ++t)
    c[t] = (ks >= 0 && t < d) ? alpha * static_cast<float>(cb_elem(C, ct, ks, d, t)) : 0.0f;
  u16x8 p1, p2, pn;
  float N = 0.0f;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    N = N + c[t] * c[t];
    const uint16_t h1 = f16_bits(c[t]);
    p1[t] = h1;
    p2[t] = f16_bits(c[t] - f16_val(h1));
    pn[t] = 0;
  }
  if (ks >= 0) {
    const float v = N * 0x1p-12f;
    const uint16_t n1 = f16_bits(v);
    const float r1 = v - f16_val(n1);
    const uint16_t n2 = f16_bits(r1);
    pn[0] = n1;
    pn[1] = n2;
    pn[2] = f16_bits(r1 - f16_val(n2));
  } else {
    pn[0] = 0x7c00;  // +inf: padding never wins
  }
  uint16_t* tile = apack + (k >> 5) * kS32TileHalves + (k & 31) * 8;
  *reinterpret_cast<u16x8*>(tile) = p1;
  *reinterpret_cast<u16x8*>(tile + 256) = p2;
  *reinterpret_cast<u16x8*>(tile + 512) = pn;
}

// ONE (bf16 rows against a bf16 codebook): every scaled element is exact in fp16 (bf16 has fewer
// significand bits and the power-of-two scale only moves the exponent; values that land below the
// fp16 normal range are covered by the underflow terms of the bound), so c2 = x2 = 0 and the
// second MFMA alone, (c1|N).(x1|2^12), forms alpha^2 s: one v_mfma_f32_32x32x16_f16 per tile.
// LIST: the rows are list[0 .. *list_n), and results go to their list positions (the second screen
// of the rows the first one left uncertain).
// QS (LIST only): the four waves of a block share their rows and split the codebook (few listed rows).
// PRUNE, first screen: rows in key order (pd.rord), results at the key positions, chunks visited
// outward from the wave's key and skipped when outside every row's band (see PruneData).
// PRUNE with LIST (second screen after a pruned first one): the listed rows are in key order and each
// has an exact upper bound on its best distance from the first screen (pd.lD), so the bands are fixed
// from the start; the chunks meeting them are listed once and screened in order (QS: every fourth
// to each wave).
// corder (when the codebook is packed in key order): sorted position -> codeword.
template <int CB, int NC, bool ONE, bool LIST, bool QS = false, bool PRUNE = false>
__global__ __launch_bounds__(256) void screen32_kernel(RowSrc src, const uint16_t* apack,
                                                       const float* __restrict__ alpha_p, int64_t tiles, int64_t tps,
                                                       const void* __restrict__ C, int ct, int64_t K,
                                                       float* __restrict__ pR, double* __restrict__ pD,
                                                       int* __restrict__ pK, double* __restrict__ xn2o,
                                                       float* __restrict__ xeo,
                                                       const int* __restrict__ list, const int* __restrict__ list_n,
                                                       const int* __restrict__ corder, PruneData pd, double bacc,
                                                       double bsplit) {
  constexpr bool PRUNE1 = PRUNE && !LIST, PRUNE2 = PRUNE && LIST;
  static_assert(!PRUNE1 || (ONE && !QS), "the first screen's pruning walks rows of its own");
  static_assert(!PRUNE2 || !ONE, "the pruned list screen is the split form");
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int j = lane & 31;
  const int h = lane >> 5;
  const int split = blockIdx.y;
  const int64_t ns = src.n;                      // stride of the per-split outputs
  const int64_t n = LIST ? *list_n : src.n;      // rows to screen
  const int d = src.d;
  // QS: the four waves of a block take the same 32 CB rows, each a quarter of the split's tiles, and
  // merge through LDS at the end (when the listed rows are few, rows alone would leave most SIMDs
  // idle).  Otherwise every wave has rows of its own.
  static_assert(LIST || !QS, "the shared-row split is for listed rows");
  // PRUNE: blocks take the key order from its upper end, where the bands are widest, so that the
  // longest waves start first
  const int64_t bx = PRUNE1 ? static_cast<int64_t>(gridDim.x) - 1 - blockIdx.x : static_cast<int64_t>(blockIdx.x);
  const int64_t row0 = QS ? static_cast<int64_t>(blockIdx.x) * (32 * CB)
                          : (bx * 4 + wave) * (32 * CB);
  if (row0 >= n) return;  // uniform over the block in QS mode; the only barrier is below
  const float alpha = alpha_p[0];
  __shared__ double sD[QS ? 4 : 1][QS ? 32 * CB : 1];
  __shared__ int sK[QS ? 4 : 1][QS ? 32 * CB : 1];
  __shared__ float sR[QS ? 4 : 1][QS ? 32 * CB : 1];
  // PRUNE: per row alpha ||x||, alpha x_j, alpha x_q and the scaled D_up offset (negative: the row
  // takes no part); per wave the lists of chunks above and below its start
  __shared__ float sBand[PRUNE1 ? 4 : 1][PRUNE1 ? CB : 1][4][32];
  __shared__ uint16_t sList[PRUNE ? 4 : 1][PRUNE1 ? 2 : 1][PRUNE ? 1024 : 1];
  // PRUNE2: the wave's union band, as float bounds {lo1, hi1, lo2, hi2} in the scaled units
  float blo1 = __builtin_inff(), bhi1 = -__builtin_inff(), blo2 = __builtin_inff(), bhi2 = -__builtin_inff();
  float blo3 = __builtin_inff(), bhi3 = -__builtin_inff();

  h8 b1[CB], b2[CB];
  bool forced[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int64_t i = row0 + cb * 32 + j;
    const bool ok = i < n;
    float v[8];
    const int64_t off = ok ? row_offset(src, LIST ? list[i] : (PRUNE1 ? pd.rord[i] : i)) : 0;
    if (src.type == ET_F32) {
      load_f32_elems<8>(static_cast<const float*>(src.base) + off, d, ok, v);
    } else if (src.type == ET_BF16) {
      load_bf16_elems<8>(static_cast<const uint16_t*>(src.base) + off, d, ok, v);
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t) v[t] = (ok && t < d) ? static_cast<float>(row_elem(src, off, t)) : 0.0f;
    }
    bool over = false;
    float xs[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      xs[t] = alpha * (-2.0f * v[t]);
      over = over || !(fabsf(xs[t]) < 65504.0f);
    }
    u16x8 p1, p2;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float x = over ? 0.0f : xs[t];
      const uint16_t x1 = f16_bits(x);
      p1[t] = x1;
      p2[t] = h ? static_cast<uint16_t>(t < 3 ? 0x6c00 : 0)  // 0x6c00 = 2^12
                : (ONE ? x1 : f16_bits(x - f16_val(x1)));
    }
    if (ONE && xeo && h == 0 && ok && split == 0) {
      // The screen on fp16-rounded operands (scaled: a = alpha c and y = -2 alpha x exactly, a = a1 + a2,
      // y = y1 + y2) drops sum_t a_t y2_t + sum_t a2_t y1_t per codeword, with |a2_t| <= 2^-11 |a_t|
      // (elements below the fp16 normal range: the bound's underflow terms).  For ||c|| <= R that is at
      // most R (||y2|| + 2^-11 (1 + 2^-11) ||y||) / alpha: the row's own remainder instead of its worst
      // case 2^-11 ||y|| (on average about 0.4 of it).  fp64 rows add the rounding of x to fp32,
      // 2^-24 ||y|| / alpha.  The fp32 sums err far less than the 2^-9 margin.
      float y2s = 0.0f, ys = 0.0f;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float y2 = over ? 0.0f : xs[t] - f16_val(p1[t]);
        y2s = y2s + y2 * y2;
        ys = ys + xs[t] * xs[t];
      }
      const float ny = sqrtf(ys);
      const float e = sqrtf(y2s) + 0x1p-11f * (1.0f + 0x1p-11f) * ny + (src.type == ET_F64 ? 0x1p-23f * ny : 0.0f);
      xeo[i] = over ? 0.0f : (e / alpha) * (1.0f + 0x1p-9f);
    }
    b1[cb] = __builtin_bit_cast(h8, p1);
    b2[cb] = __builtin_bit_cast(h8, p2);
    forced[cb] = over;
    if (PRUNE2 && h == 0 && ok && !over) {
      // |x|, x_j and x_q exactly (fp64) and the first screen's exact distance (rounded up): every
      // codeword that can tie or beat it lies within sqrt(D) of them; bounds rounded outward with
      // 2^-20 relative and 2^-10 absolute margins in the scaled units
      double xn2 = 0.0, xj = 0.0, xq = 0.0;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        xn2 = xn2 + static_cast<double>(v[t]) * static_cast<double>(v[t]);
        xj = (t == pd.jp) ? static_cast<double>(v[t]) : xj;
        xq = (t == pd.jq) ? static_cast<double>(v[t]) : xq;
      }
      const double a = static_cast<double>(alpha);
      const double An = sqrt(xn2) * a, Pj = xj * a, Qq = xq * a;
      const double r = sqrt(static_cast<double>(pd.lD[i])) * a;
      const double m1 = 0x1p-20 * (An + r) + 0x1p-10, m2 = 0x1p-20 * (fabs(Pj) + r) + 0x1p-10;
      const double m3 = 0x1p-20 * (fabs(Qq) + r) + 0x1p-10;
      blo1 = fminf(blo1, f32_down_any(An - r - m1));
      bhi1 = fmaxf(bhi1, f32_up_any(An + r + m1));
      blo2 = fminf(blo2, f32_down_any(Pj - r - m2));
      bhi2 = fmaxf(bhi2, f32_up_any(Pj + r + m2));
      blo3 = fminf(blo3, f32_down_any(Qq - r - m3));
      bhi3 = fmaxf(bhi3, f32_up_any(Qq + r + m3));
    }
    if (PRUNE1 && h == 0) {
      // the row's band terms in units of alpha: ||x||, x_j and x_q exactly (fp64), and
      // D_up - m = alpha^2 ||x||^2 + alpha^2 delta(R = max ||c||), rounded up
      double xn2 = 0.0, xj = 0.0, xq = 0.0;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        xn2 = xn2 + static_cast<double>(v[t]) * static_cast<double>(v[t]);
        xj = (t == pd.jp) ? static_cast<double>(v[t]) : xj;
        xq = (t == pd.jq) ? static_cast<double>(v[t]) : xq;
      }
      const double a = static_cast<double>(alpha);
      const double An = sqrt(xn2) * a, cm = static_cast<double>(pd.prm[3]);
      const double B = a * a * xn2 + bacc * 0x1p-24 * (cm * cm + 2.0 * An * cm) + bsplit * An * cm +
                       0x1p-24 * 2.8285 * (cm + 2.0 * An) + 0x1p-12;
      sBand[wave][cb][0][j] = static_cast<float>(An);
      sBand[wave][cb][1][j] = static_cast<float>(xj * a);
      sBand[wave][cb][2][j] = static_cast<float>(xq * a);
      sBand[wave][cb][3][j] = (ok && !over) ? f32_up(B) * (1.0f + 0x1p-20f) : -1.0f;
    }
  }

  float m[CB], rest[CB], cm[CB];
  int id[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    m[cb] = __builtin_inff();
    rest[cb] = __builtin_inff();
    cm[cb] = __builtin_inff();
    id[cb] = -1;
  }

  int64_t t0 = static_cast<int64_t>(split) * tps;
  int64_t t1 = (t0 + tps < tiles) ? t0 + tps : tiles;
  if (QS && !PRUNE2) {
    const int64_t q = (t1 - t0 + 7) / 8 * 2;  // even shares: chunks of two tiles stay aligned
    const int64_t a = t0 + __builtin_amdgcn_readfirstlane(wave) * q;  // wave-uniform: scalar bounds
    t1 = (a + q < t1) ? a + q : t1;
    t0 = a;
  }
  if (t0 < t1) {
    // Codebook tiles come in through a buffer resource: the per-lane byte offset is fixed, the
    // tile offset is a scalar, so a tile costs no vector address arithmetic.  Lanes 0-31 read c1
    // twice, lanes 32-63 read c2 and the N terms.  (Tile indices fit in 32 bits.)
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(apack), 0, static_cast<int>(tiles * kS32TileHalves * 2), 0x00020000);
    const int voff1 = (j * 8 + h * 256) * 2, voff2 = (j * 8 + h * 512) * 2;
    const int T0 = static_cast<int>(t0), T1 = static_cast<int>(t1);
    auto load = [&](int T, h8& a1, h8& a2) {
      if (!ONE)
        a1 = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rs, voff1, T * (kS32TileHalves * 2), 0));
      a2 = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rs, voff2, T * (kS32TileHalves * 2), 0));
    };
    // Software-pipelined over the column blocks: the MFMA pair of block cb is issued before the
    // minimum of block cb - 1 is folded (a depth-3 v_min3 tree), so a wave keeps the matrix core
    // and the VALU busy at the same time.  The first tile of a chunk starts its minimum afresh.
    auto tile = [&](const h8& a1, const h8& a2, bool first) {
      f16v acc[2];
#pragma unroll
      for (int cb = 0; cb <= CB; ++cb) {
        if (cb < CB) {
          f16v z = {};
          if (ONE) {
            acc[cb & 1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a2, b2[cb], z, 0, 0, 0);
          } else {
            acc[cb & 1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a1, b1[cb], z, 0, 0, 0);
            acc[cb & 1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a2, b2[cb], acc[cb & 1], 0, 0, 0);
          }
        }
        if (cb > 0) {
          const f16v& a = acc[(cb - 1) & 1];
          cm[cb - 1] = first ? min_fold16(a[0], a) : min_fold16(cm[cb - 1], a);
        }
        if (CRVQ_S32_SCHED) {
          if (cb < CB) __builtin_amdgcn_sched_group_barrier(0x008, ONE ? 1 : 2, 0);
          if (cb > 0) __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
        }
      }
    };
    auto fold = [&](int Ci) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        rest[cb] = __builtin_amdgcn_fmed3f(m[cb], rest[cb], cm[cb]);
        const bool lt = cm[cb] < m[cb];
        m[cb] = fminf(m[cb], cm[cb]);
        id[cb] = lt ? Ci : id[cb];
      }
    };
    static_assert(NC == 1 || NC == 2, "chunks of one or two tiles");
    static_assert(!PRUNE || NC == 2, "pruning works on chunks of two tiles");
    if constexpr (PRUNE2) {
      // the wave's band (its rows' union), then the chunks of the split's range that meet it, listed
      // in LDS in ascending order; the loads of the next chunk are issued before the current one's MFMAs
#pragma unroll
      for (int sh = 1; sh < 64; sh <<= 1) {
        blo1 = fminf(blo1, __shfl_xor(blo1, sh));
        bhi1 = fmaxf(bhi1, __shfl_xor(bhi1, sh));
        blo2 = fminf(blo2, __shfl_xor(blo2, sh));
        bhi2 = fmaxf(bhi2, __shfl_xor(bhi2, sh));
        blo3 = fminf(blo3, __shfl_xor(blo3, sh));
        bhi3 = fmaxf(bhi3, __shfl_xor(bhi3, sh));
      }
      PruneCursor cur = {0, 0, 0, 0, 0, rfl(okey(blo1)), rfl(okey(bhi1)), rfl(okey(blo2)), rfl(okey(bhi2)),
                         rfl(okey(blo3)), rfl(okey(bhi3))};
      const int c0 = static_cast<int>(t0 >> 1), c1 = static_cast<int>(t1 >> 1);
      uint16_t* Lc = &sList[wave][0][0];
      int cnt = 0;
      const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
      for (int cb0 = c0; cb0 < c1; cb0 += 64) {
        const int c = cb0 + lane;
        const int cs = c < c1 ? c : c0;
        const bool keep = c < c1 && prune_keep(pd.cbnd[cs], pd.cbnd3[cs], cur);
        const uint64_t km = __ballot(keep);
        if (keep) Lc[cnt + __popcll(km & lt)] = static_cast<uint16_t>(c);
        cnt += __popcll(km);
      }
      cnt = static_cast<int>(rfl(static_cast<uint32_t>(cnt)));
      const int step = QS ? 4 : 1;
      int li = QS ? static_cast<int>(rfl(static_cast<uint32_t>(wave))) : 0;
      auto next = [&]() {
        const int c = li < cnt ? static_cast<int>(rfl(Lc[li])) : -1;
        li += step;
        return c;
      };
      h8 qa1, qa2, qb1, qb2;
      int Cc = next();
      int Cn = Cc >= 0 ? next() : -1;
      if (Cc >= 0) {
        load(2 * Cc, qa1, qa2);
        load(2 * Cc + 1, qb1, qb2);
      }
      while (Cc >= 0) {
        const int Tn = Cn >= 0 ? 2 * Cn : 2 * Cc;
        tile(qa1, qa2, true);
        load(Tn, qa1, qa2);
        // the first tile's minima are complete before the second tile's matrix products start (left
        // to the compiler, both tiles' accumulators were live at once: twice the registers)
        if (CRVQ_PRUNE2_SB) {
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) __asm__ volatile("" : "+v"(cm[cb]));
          __builtin_amdgcn_sched_barrier(0);
        }
        tile(qb1, qb2, false);
        if (CRVQ_PRUNE2_SB) {
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) __asm__ volatile("" : "+v"(cm[cb]));
        }
        fold(2 * Cc);
        load(Tn + 1, qb1, qb2);
        Cc = Cn;
        Cn = Cn >= 0 ? next() : -1;
      }
    } else if constexpr (PRUNE1) {
      // Chunks (tile pairs) from the wave's key outward, alternately above and below; a side stops
      // where the envelope leaves the norm band, a chunk is skipped when outside either band.  The
      // bands start open and narrow as the running minima fall (recomputed after 4, 8, 16, ...
      // chunks).  All of this is wave-uniform control on the scalar unit.
      const int c0 = static_cast<int>(t0 >> 1), c1 = static_cast<int>(t1 >> 1);
      const int64_t mid = (row0 + 64 < n) ? row0 + 64 : n - 1;
      // (readfirstlane: the wave index is uniform, which the compiler cannot see)
      int cc = __builtin_amdgcn_readfirstlane(pd.coff[pd.rkey[pd.rord[mid]]] >> 6);
      cc = cc < c0 ? c0 : (cc >= c1 ? c1 - 1 : cc);
      PruneCursor cur = {0, c1 - cc, 0, cc - c0, 0, 0u, 0xffffffffu, 0u, 0xffffffffu, 0u, 0xffffffffu};
      uint16_t* Ul = &sList[wave][0][0];
      uint16_t* Dl = &sList[wave][1][0];
      for (int i = lane; i < cur.un; i += 64) Ul[i] = static_cast<uint16_t>(cc + i);
      for (int i = lane; i < cur.dn; i += 64) Dl[i] = static_cast<uint16_t>(cc - 1 - i);
      // The chunk after next is chosen at the end of an iteration, so the body (MFMAs, minimum
      // folds, the next chunk's loads) stays straight-line; past the last chunk the loads repeat
      // a valid tile and are not used.
      int done = 0, at = CRVQ_PRUNE_FIRST;
      auto renew = [&]() {
        if (++done == at) {
          prune_band<CB>(cur, m, &sBand[wave][0][0][0], j);
          // chunks already taken stay; the rest is filtered
          cur.un = prune_filter(Ul, cur.ui, cur.un, true, cur, pd, lane);
          cur.dn = prune_filter(Dl, cur.di, cur.dn, false, cur, pd, lane);
          cur.ui = 0;
          cur.di = 0;
          at = at < CRVQ_PRUNE_CAP ? 2 * at : at + CRVQ_PRUNE_CAP;
        }
      };
      h8 qa, qb;
      int Cc = prune_take(cur, Ul, Dl);
      int Cn = Cc >= 0 ? prune_take(cur, Ul, Dl) : -1;
      if (Cc >= 0) {
        load(2 * Cc, qa, qa);
        load(2 * Cc + 1, qb, qb);
      }
      while (Cc >= 0) {
        const int Tn = Cn >= 0 ? 2 * Cn : 2 * Cc;
        tile(qa, qa, true);
        load(Tn, qa, qa);
        tile(qb, qb, false);
        fold(2 * Cc);
        load(Tn + 1, qb, qb);
        renew();
        Cc = Cn;
        Cn = Cn >= 0 ? prune_take(cur, Ul, Dl) : -1;
      }
    } else {
    // Two tiles per iteration from two register sets; each set is refilled right after its MFMAs,
    // one iteration ahead of its next use.
    h8 qa1, qa2, qb1, qb2;
    load(T0, qa1, qa2);
    load((T0 + 1 < T1) ? T0 + 1 : T1 - 1, qb1, qb2);
    int T = T0;
    for (; T + 2 <= T1; T += 2) {
      tile(qa1, qa2, true);
      if (NC == 1) fold(T);
      load((T + 2 < T1) ? T + 2 : T1 - 1, qa1, qa2);
      tile(qb1, qb2, NC == 1);
      fold(NC == 1 ? T + 1 : T);
      load((T + 3 < T1) ? T + 3 : T1 - 1, qb1, qb2);
    }
    if (T < T1) {
      tile(qa1, qa2, true);
      fold(T);
    }
    }
  }

  // The lane half with the smaller kept-chunk minimum wins the row; the other half's best chunk
  // joins the bound.  The winner half's 16 codewords of every tile of the kept chunk are re-scored
  // exactly, 8 per lane half, and reduced in (D, k) order.
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int64_t i = row0 + cb * 32 + j;
    const bool valid = i < n;
    // the row's index in the source; results go to the row's position i (list or key order)
    const int64_t pi = (LIST && valid) ? list[i] : ((PRUNE1 && valid) ? pd.rord[i] : i);
    const int64_t oi = i;
    const float mg = m[cb];
    const float om = __shfl_xor(mg, 32);
    const int hw = (om < mg || (om == mg && h == 1)) ? 1 - h : h;
    float rr = (h == hw) ? rest[cb] : fminf(rest[cb], mg);
    rr = fminf(rr, __shfl_xor(rr, 32));
    if (forced[cb]) rr = -__builtin_inff();
    const int Tw = __shfl(id[cb], j + 32 * hw);
    double xd[8];
    load_row_exact<8>(src, pi, valid, xd);
    double D = __builtin_inf();
    int kk = INT_MAX;
#pragma unroll
    for (int u = 0; u < NC; ++u) {
      const int64_t T = static_cast<int64_t>(Tw) + u;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        // codewords 8 (2 h + q) + 4 hw + s, s = 0..3, of the tile
        const int64_t k0 = T * kS32Tile + 8 * (2 * h + q) + 4 * hw;
        float cw[4][8];
        bool ok[4];
        int64_t ko[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          ok[s] = valid && Tw >= 0 && T < t1 && k0 + s < K;
          ko[s] = (corder && ok[s]) ? static_cast<int64_t>(corder[k0 + s]) : k0 + s;
          ok[s] = ok[s] && ko[s] >= 0 && ko[s] < K;
          load_codeword<8>(C, ct, ko[s], d, ok[s], cw[s]);
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          if (ok[s]) {
            double Du = 0.0;
#pragma unroll
            for (int t = 0; t < 8; ++t) {
              if (t < d) {
                const double diff = xd[t] - static_cast<double>(cw[s][t]);
                Du = Du + diff * diff;
              }
            }
            const int ku = static_cast<int>(ko[s]);
            if (cless(Du, ku, D, kk)) {
              D = Du;
              kk = ku;
            }
          }
        }
      }
    }
    const double oD = __shfl_xor(D, 32);
    const int ok2 = __shfl_xor(kk, 32);
    if (cless(oD, ok2, D, kk)) {
      D = oD;
      kk = ok2;
    }
    if (QS) {
      if (h == 0) {
        sD[wave][cb * 32 + j] = D;
        sK[wave][cb * 32 + j] = kk;
        sR[wave][cb * 32 + j] = rr;
      }
      if (h == 0 && valid && wave == 0 && split == 0) {
        double xn2 = 0.0;
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (t < d) xn2 = xn2 + xd[t] * xd[t];
        xn2o[i] = xn2;
      }
    } else if (h == 0 && valid) {
      double xn2 = 0.0;
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (t < d) xn2 = xn2 + xd[t] * xd[t];
      pD[static_cast<int64_t>(split) * ns + oi] = D;
      pK[static_cast<int64_t>(split) * ns + oi] = kk;
      pR[static_cast<int64_t>(split) * ns + oi] = rr;
      if (split == 0) xn2o[oi] = xn2;
    }
  }
  if (QS) {
    // merge the four quarters as splits are merged: the (D, k)-smallest exact winner, the smallest rest
    __syncthreads();
    for (int r = threadIdx.x; r < 32 * CB; r += 256) {
      const int64_t i = row0 + r;
      if (i >= n) continue;
      double D = sD[0][r];
      int kk = sK[0][r];
      float rr = sR[0][r];
#pragma unroll
      for (int w = 1; w < 4; ++w) {
        if (cless(sD[w][r], sK[w][r], D, kk)) {
          D = sD[w][r];
          kk = sK[w][r];
        }
        rr = fminf(rr, sR[w][r]);
      }
      pD[static_cast<int64_t>(split) * ns + i] = D;
      pK[static_cast<int64_t>(split) * ns + i] = kk;
      pR[static_cast<int64_t>(split) * ns + i] = rr;
    }
  }
}

// ------------------------------------------------------------------------------------------------
// 4. merge the splits, certify, emit; rescue the uncertain rows exactly
// ------------------------------------------------------------------------------------------------
// Finalize, one thread per row.  Top-1: merge the splits' exact winners.  Top-B: re-score in fp64
// the four codewords of every kept tile of every lane group and split.  Then order by (D, k) and
// certify against the screen bound.
// Screen error bound (certification): delta = acc_ulps 2^-24 (R^2 + 2 ||x|| R) + split_coef ||x|| R
// + abs_coef (||x|| + R + 1), with R = ||x|| + sqrt(D_top).  A scaled screen (alpha != null) stores
// alpha^2 s: its bound values are divided by alpha^2 and the fp16 underflow terms
// 2^-24 sqrt(8) (R + 2 ||x||) / alpha + 2^-12 / alpha^2 are added.
struct ScreenBound {
  double acc_ulps;
  double split_coef;
  double abs_coef;
  const float* alpha;
  const float* row_e;  // when set: per row (position) the split term's factor of R, replacing split_coef ||x||
};

// Writes a row's result: its code and distance (top-1) or its sorted (D, k) list, padded with
// (+inf, -1) past the codebook size.
template <int NB>
__device__ __forceinline__ void emit_row(int64_t row, const double (&ED)[NB], const int (&EK)[NB], int top, int need,
                                         int32_t* codes, float* dist, double* rowD, int* rowK) {
  // INT_MAX: no codeword compared below +inf (a row with a NaN element); the code is then 0, a
  // defined in-range value, and the distance NaN
  if (codes) {
    const bool none = EK[0] == INT_MAX;
    codes[row] = none ? 0 : EK[0];
    // (the NaN as a bit pattern: this file is compiled without NaN semantics)
    if (dist) dist[row] = none ? __uint_as_float(0x7fc00000u) : static_cast<float>(ED[0]);
  } else {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (j < top) {
        const bool real = j < need;
        rowD[row * top + j] = real ? ED[j] : __builtin_inf();
        rowK[row * top + j] = real ? (EK[j] == INT_MAX ? 0 : EK[j]) : -1;
      }
    }
  }
}

// One thread per row; rows that fail the certification are appended to the rescue list.
template <int KS, int NB>
__global__ __launch_bounds__(256) void finalize_kernel(RowSrc src, int splits, int chunk, int64_t tps, int64_t tiles,
                                                       int top, const int* __restrict__ pT,
                                                       const float* __restrict__ pM,
                                                       const float* __restrict__ pR, const double* __restrict__ pD,
                                                       const int* __restrict__ pK, const double* __restrict__ xn2a,
                                                       const void* __restrict__ C, int ct, int64_t K,
                                                       ScreenBound bound, int* __restrict__ rcount,
                                                       int* __restrict__ rlist, int32_t* __restrict__ codes,
                                                       float* __restrict__ dist, double* __restrict__ rowD,
                                                       int* __restrict__ rowK) {
  constexpr int DM = 4 * KS;  // dimensions this instantiation covers (d <= DM)
  const int tid = threadIdx.x;
  const int64_t n = src.n;
  const int d = src.d;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + tid;
  const bool valid = i < n;
  const int need = static_cast<int>((top < K) ? top : K);

  double xd[DM];
  double xn2 = 0.0;
  if constexpr (NB > 1) {
    load_row_exact<DM>(src, i, valid, xd);
#pragma unroll
    for (int t = 0; t < DM; ++t)
      if (t < d) xn2 = xn2 + xd[t] * xd[t];
  }

  double LD[NB];
  int LK[NB];
  float rest = __builtin_inff();
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    LD[j] = __builtin_inf();
    LK[j] = INT_MAX;
  }
  bool certain = false;
  if (valid && NB == 1) {
    xn2 = xn2a[i];
    for (int s = 0; s < splits; ++s) {
      const double D = pD[static_cast<int64_t>(s) * n + i];
      const int k = pK[static_cast<int64_t>(s) * n + i];
      if (cless(D, k, LD[0], LK[0])) {
        LD[0] = D;
        LK[0] = k;
      }
      rest = fminf(rest, pR[static_cast<int64_t>(s) * n + i]);
    }
  }
  if (valid) {
    // Top-B: only kept tiles whose screen minimum is within a small margin of the top-th smallest
    // kept minimum can hold one of the top answers in practice; the others are not re-scored and
    // their minima join "rest", so the certificate below stays exact (a row whose answer lies in
    // a skipped tile fails it and is rescued).
    float thr = __builtin_inff();
    // the first split's kept minima stay in registers from the threshold to the selection (with one
    // split, the usual case, pM is read once; the kept tile ids only for the tiles re-scored)
    float pm0[NB > 1 ? 4 : 1][NB];
    if (NB > 1 && valid) {
      // the NB smallest kept tile minima, ascending: each lane group's list is ascending already, so
      // it is merged in (the smaller of the running list and the group's taken in reverse is a
      // bitonic sequence holding the NB smallest of both; a half-cleaner network sorts it)
      float sm[NB];
#pragma unroll
      for (int j = 0; j < NB; ++j) sm[j] = __builtin_inff();
      for (int s = 0; s < splits; ++s) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float b[NB];
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            b[j] = pM[((static_cast<int64_t>(s) * 4 + g) * NB + j) * n + i];
            if (s == 0) pm0[g][j] = b[j];
          }
#pragma unroll
          for (int j = 0; j < NB; ++j) sm[j] = fminf(sm[j], b[NB - 1 - j]);
#pragma unroll
          for (int w = NB / 2; w >= 1; w >>= 1) {
#pragma unroll
            for (int j = 0; j < NB; ++j) {
              if ((j & w) == 0) {
                const float lo = fminf(sm[j], sm[j + w]), hi = fmaxf(sm[j], sm[j + w]);
                sm[j] = lo;
                sm[j + w] = hi;
              }
            }
          }
        }
      }
      float mt = sm[0];
#pragma unroll
      for (int q = 0; q < NB; ++q)
        if (q == need - 1) mt = sm[q];
      thr = mt + 0x1p-12f * (fabsf(mt) + static_cast<float>(xn2));
    }
    // The kept tiles to re-score, as a bit set over the (group, slot) pairs, so that a wave loops over
    // the most any of its rows needs (typically a handful) instead of every kept slot; the others'
    // minima bound their codewords and join "rest".  A slot holding no tile has the minimum +inf: it
    // joins neither (nor does it below, where its tile id is negative).  The first split's set is
    // taken here, from the minima in registers.
    uint64_t todo0 = 0;
    if (NB > 1) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const float mj = pm0[g][j];
          if (mj <= thr)
            todo0 |= uint64_t{1} << (g * NB + j);
          else
            rest = fminf(rest, mj);
        }
      }
    }
    for (int s = 0; s < (NB > 1 ? splits : 0); ++s) {
      rest = fminf(rest, pR[static_cast<int64_t>(s) * n + i]);
      uint64_t todo = todo0;
      if (s > 0) {
        todo = 0;
        for (int g = 0; g < 4; ++g) {
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const float mj = pM[((static_cast<int64_t>(s) * 4 + g) * NB + j) * n + i];
            if (mj <= thr)
              todo |= uint64_t{1} << (g * NB + j);
            else
              rest = fminf(rest, mj);
          }
        }
      }
      const int64_t ts1 = (static_cast<int64_t>(s) + 1) * tps < tiles ? (static_cast<int64_t>(s) + 1) * tps : tiles;
      while (todo) {
        const int q = __builtin_ctzll(todo);
        todo &= todo - 1;
        const int g = q / NB, j = q - (q / NB) * NB;
        const int T0 = pT[((static_cast<int64_t>(s) * 4 + g) * NB + j) * n + i];
        if (T0 < 0) continue;  // an empty slot (the threshold is +inf)
        for (int u = 0; u < chunk && T0 + u < ts1; ++u) {  // the kept tile, or every tile of its chunk
          const int T = T0 + u;
          float cw[4][DM];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int64_t k = static_cast<int64_t>(T) * 16 + 4 * g + r;
            load_codeword<DM>(C, ct, k, d, k < K, cw[r]);
          }
          if constexpr (NB >= 4) {
            double Dc[4];
            int Kc[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int64_t k = static_cast<int64_t>(T) * 16 + 4 * g + r;
              double acc = 0.0;
#pragma unroll
              for (int t = 0; t < DM; ++t) {
                if (t < d) {
                  const double diff = xd[t] - static_cast<double>(cw[r][t]);
                  acc = acc + diff * diff;
                }
              }
              Dc[r] = k < K ? acc : __builtin_inf();  // past the book: never taken
              Kc[r] = k < K ? static_cast<int>(k) : INT_MAX;
            }
            list_merge4<NB>(LD, LK, Dc, Kc);
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int64_t k = static_cast<int64_t>(T) * 16 + 4 * g + r;
              if (k < K) {
                double acc = 0.0;
#pragma unroll
                for (int t = 0; t < DM; ++t) {
                  if (t < d) {
                    const double diff = xd[t] - static_cast<double>(cw[r][t]);
                    acc = acc + diff * diff;
                  }
                }
                list_insert<NB>(LD, LK, acc, static_cast<int>(k));
              }
            }
          }
        }
      }
    }
    double Dl = LD[0];
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if (j == need - 1) Dl = LD[j];
    if (rest == __builtin_inff()) {
      certain = true;  // every codeword was scored exactly
    } else {
      const double xn = sqrt(xn2);
      const double R = xn + sqrt(Dl);
      double delta = bound.acc_ulps * 0x1p-24 * (R * R + 2.0 * xn * R) + bound.split_coef * xn * R +
                     bound.abs_coef * (xn + R + 1.0) + 1e-35;
      double restd = static_cast<double>(rest);
      if (bound.alpha) {
        const double inv = 1.0 / static_cast<double>(bound.alpha[0]);
        restd = restd * inv * inv;
        delta += 0x1p-24 * 2.8285 * (R + 2.0 * xn) * inv + 0x1p-12 * inv * inv;
      }
      certain = Dl < restd + xn2 - delta;
    }
  }

  // An uncertain row is written with its tentative result (the rescue starts from that exact
  // distance) and goes to the rescue list; its order there does not affect any result.
  if (valid) emit_row<NB>(i, LD, LK, top, need, codes, dist, rowD, rowK);
  list_append(valid && !certain, i, rcount, rlist);
}

// Fast forms of the small-codebook kernel: FT 1 = fp32 rows packed back to back (d = 8, 16-byte
// aligned) against an fp32 codebook, FT 2 = bf16 rows packed back to back (d = 8, 16-byte aligned)
// against a bf16 codebook; FT 0 = any layout and type.  Row i and codeword k of a fast form are one
// 32- or 16-byte load at a fixed stride.
template <int FT>
__device__ __forceinline__ void small1_row(const void* base, int64_t i, float (&v)[8]) {
  if constexpr (FT == 1) {
    const f4* p = static_cast<const f4*>(base) + 2 * i;
    const f4 a = p[0], b = p[1];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      v[t] = a[t];
      v[4 + t] = b[t];
    }
  } else {
    const uint4 q = static_cast<const uint4*>(base)[i];
    const uint32_t u[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      v[2 * t] = __uint_as_float(u[t] << 16);
      v[2 * t + 1] = __uint_as_float(u[t] & 0xffff0000u);
    }
  }
}

// The fast form that applies to these rows and this codebook (0 when none does).
int small1_form(const RowSrc& src, const void* C, int ct) {
  if (src.d != 8 || src.ld != src.vpr * 8) return 0;
  const uintptr_t a = reinterpret_cast<uintptr_t>(src.base) | reinterpret_cast<uintptr_t>(C);
  if ((a & 15) != 0) return 0;
  if (src.type == ET_F32 && ct == ET_F32) return 1;
  if (src.type == ET_BF16 && ct == ET_BF16) return 2;
  return 0;
}

// Top-1 against a small codebook (at most 16 tiles of 16, one split): the split-bf16 screen of
// screen_kernel, tracked per cell.  A cell is the four codewords 16 T + 4 g .. 16 T + 4 g + 3 whose
// screen values one MFMA tile T gives lane group g for a row; every lane keeps, per row, the smallest
// cell minimum with the cell's first codeword and the second smallest cell minimum (two VALU
// operations per four values for the cell minimum, four per cell for the tracking).  After the four
// lane groups of a row are merged, the four codewords of the row's winning cell are scored exactly in
// fp64 and taken in (D, k) order; the winner is certified against the smallest screen value outside
// that cell with the same bound as finalize_kernel (R = ||x|| + sqrt(D)).  The row's result is
// written directly (codes / dist, or rowD / rowK for a beam step); an uncertain row keeps it as its
// tentative result and is appended to the rescue list.
template <int CB, int FT>
__global__ __launch_bounds__(256) void screen_small1_kernel(RowSrc src, const void* __restrict__ apack,
                                                            const float* __restrict__ cnp, int64_t tiles,
                                                            const void* __restrict__ C, int ct, int64_t K,
                                                            ScreenBound bound, int* __restrict__ rcount,
                                                            int* __restrict__ rlist, int32_t* __restrict__ codes,
                                                            float* __restrict__ dist, double* __restrict__ rowD,
                                                            int* __restrict__ rowK) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int jl = lane & 15;
  const int g = lane >> 4;
  const int64_t n = src.n;
  const int d = src.d;
  const int64_t row0 = (static_cast<int64_t>(blockIdx.x) * 4 + wave) * (16 * CB);
  if (row0 >= n) return;  // no barriers below
  const int dd = FT ? 8 : d;
  SplitOps::B bop[CB];
  if constexpr (FT == 0) {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int64_t i = row0 + cb * 16 + jl;
      bop[cb] = SplitOps::make_b(src, i, i < n, g);
    }
  } else {
    // every load in flight before the first split; a row past the end repeats the last row (its
    // screen column is never read)
    float v[CB][8];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int64_t i = row0 + cb * 16 + jl;
      small1_row<FT>(src.base, i < n ? i : n - 1, v[cb]);
    }
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) bop[cb] = SplitOps::make_b_vals(v[cb], g);
  }
  float m1[CB], m2[CB];
  int i1[CB];  // first codeword of the cell holding m1
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    m1[cb] = __builtin_inff();
    m2[cb] = __builtin_inff();
    i1[cb] = 0x7fffffff;
  }
  // tile T + 1's operands are loaded while tile T is screened (the last tile loads itself again)
  SplitOps::A a = SplitOps::load_a(apack, 0, lane);
  f4 c4 = *reinterpret_cast<const f4*>(cnp + 4 * g);
  for (int64_t T = 0; T < tiles; ++T) {
    const int64_t Tn = (T + 1 < tiles) ? T + 1 : T;
    const SplitOps::A an = SplitOps::load_a(apack, Tn, lane);
    const f4 c4n = *reinterpret_cast<const f4*>(cnp + Tn * 16 + 4 * g);
    const int kb = static_cast<int>(T) * 16 + 4 * g;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const f4 acc = SplitOps::mfma(a, bop[cb], c4);
      const float cm = fminf(fminf(acc[0], acc[1]), fminf(acc[2], acc[3]));
      m2[cb] = __builtin_amdgcn_fmed3f(m1[cb], m2[cb], cm);  // m1 <= m2 holds throughout
      const bool lt = cm < m1[cb];
      m1[cb] = lt ? cm : m1[cb];
      i1[cb] = lt ? kb : i1[cb];
    }
    a = an;
    c4 = c4n;
  }
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    // merge the four lane groups of the row (lanes jl, jl + 16, jl + 32, jl + 48)
#pragma unroll
    for (int sh = 16; sh <= 32; sh <<= 1) {
      const float om1 = __shfl_xor(m1[cb], sh), om2 = __shfl_xor(m2[cb], sh);
      const int oi1 = __shfl_xor(i1[cb], sh);
      const float nm2 = fminf(fminf(m2[cb], om2), fmaxf(m1[cb], om1));
      // evaluated without short-circuit, so the compiler selects instead of branching
      const bool take = (om1 < m1[cb]) | ((om1 == m1[cb]) & (oi1 < i1[cb]));
      m1[cb] = take ? om1 : m1[cb];
      i1[cb] = take ? oi1 : i1[cb];
      m2[cb] = nm2;
    }
  }
  // Every lane group now holds the merged state of all CB column blocks; lane group g finishes the
  // rows of blocks g, g + 4, ... so all 64 lanes share the exact epilogue.
#pragma unroll
  for (int rr = 0; rr < (CB + 3) / 4; ++rr) {
    float s2 = __builtin_inff();
    int k1 = 0x7fffffff;
#pragma unroll
    for (int cb = 4 * rr; cb < 4 * rr + 4 && cb < CB; ++cb) {
      if (cb - 4 * rr == g) {
        s2 = m2[cb];
        k1 = i1[cb];
      }
    }
    const int cbm = 4 * rr + g;
    const int64_t i = row0 + cbm * 16 + jl;
    if (cbm >= CB || i >= n) continue;
    // a winning cell has a screen value below +inf, so its first codeword is a real one (padding
    // codewords, past K, screen to +inf); no winner (a NaN row) leaves the row to the rescue
    const bool has = k1 >= 0 && k1 < K;
    const int kc = has ? k1 : 0;
    double xd[8];
    float cw[4][8];
    if constexpr (FT == 0) {
      load_row_exact<8>(src, i, true, xd);
#pragma unroll
      for (int r = 0; r < 4; ++r) load_codeword<8>(C, ct, kc + r, d, kc + r < K, cw[r]);
    } else {
      float v[8];
      small1_row<FT>(src.base, i, v);
#pragma unroll
      for (int r = 0; r < 4; ++r) small1_row<FT>(C, kc + r < K ? kc + r : kc, cw[r]);
#pragma unroll
      for (int t = 0; t < 8; ++t) xd[t] = static_cast<double>(v[t]);
    }
    double xn2 = 0.0;
#pragma unroll
    for (int t = 0; t < 8; ++t)
      if (t < dd) xn2 = xn2 + xd[t] * xd[t];
    double D1 = 0.0;
    int kk = kc;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      double D = 0.0;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        if (t < dd) {
          const double diff = xd[t] - static_cast<double>(cw[r][t]);
          D = D + diff * diff;
        }
      }
      if (r == 0) {
        D1 = D;
      } else if (kc + r < K && cless(D, kc + r, D1, kk)) {
        D1 = D;
        kk = kc + r;
      }
    }
    bool certain = has;
    if (certain && s2 != __builtin_inff()) {
      const double xn = sqrt(xn2);
      const double R = xn + sqrt(D1);
      const double delta = bound.acc_ulps * 0x1p-24 * (R * R + 2.0 * xn * R) + bound.split_coef * xn * R +
                           bound.abs_coef * (xn + R + 1.0) + 1e-35;
      certain = D1 < static_cast<double>(s2) + xn2 - delta;
    }
    if (codes) {
      codes[i] = kk;
      if (dist) dist[i] = static_cast<float>(D1);
    } else {
      rowD[i] = D1;
      rowK[i] = kk;
    }
    if (!certain) rlist[atomicAdd(rcount, 1)] = static_cast<int>(i);
  }
}

// Top-1 result of row `row` from its screen results at position i (splits merged in (D, k) order)
// and its certificate, written to the row's outputs; returns whether it is certain.
__device__ __forceinline__ bool finish_top1(int64_t i, int64_t row, int splits, int64_t ns,
                                            const float* __restrict__ pR, const double* __restrict__ pD,
                                            const int* __restrict__ pK, const double* __restrict__ xn2a,
                                            const ScreenBound& bound, int32_t* __restrict__ codes,
                                            float* __restrict__ dist, double* __restrict__ rowD,
                                            int* __restrict__ rowK) {
  double Dl = __builtin_inf();
  int kl = INT_MAX;
  float rest = __builtin_inff();
  for (int s = 0; s < splits; ++s) {
    const double D = pD[static_cast<int64_t>(s) * ns + i];
    const int k = pK[static_cast<int64_t>(s) * ns + i];
    if (cless(D, k, Dl, kl)) {
      Dl = D;
      kl = k;
    }
    rest = fminf(rest, pR[static_cast<int64_t>(s) * ns + i]);
  }
  bool certain;
  if (rest == __builtin_inff()) {
    certain = true;  // every codeword was scored exactly
  } else {
    const double xn2 = xn2a[i];
    const double xn = sqrt(xn2);
    const double R = xn + sqrt(Dl);
    const double sc = bound.row_e ? static_cast<double>(bound.row_e[i]) : bound.split_coef * xn;
    double delta = bound.acc_ulps * 0x1p-24 * (R * R + 2.0 * xn * R) + sc * R +
                   bound.abs_coef * (xn + R + 1.0) + 1e-35;
    double restd = static_cast<double>(rest);
    if (bound.alpha) {
      const double inv = 1.0 / static_cast<double>(bound.alpha[0]);
      restd = restd * inv * inv;
      delta += 0x1p-24 * 2.8285 * (R + 2.0 * xn) * inv + 0x1p-12 * inv * inv;
    }
    certain = Dl < restd + xn2 - delta;
  }
  if (kl == INT_MAX) {  // no score compared below +inf (a NaN element): leave it to the rescue
    kl = 0;
    certain = false;
  }
  if (codes) {
    codes[row] = kl;
    if (dist) dist[row] = static_cast<float>(Dl);
  } else {
    rowD[row] = Dl;
    rowK[row] = kl;
  }
  return certain;
}

// Top-1 finalize of the first of two screens, over every row.  A large share of rows can fail its
// wider certificate, so instead of one global counter (whose atomics serialize) each block packs its
// failing rows, in row order, into its own slice tmp[256 b ..] and writes their number to bcount[b];
// scan_counts_kernel and compact_list_kernel then build the dense list in block order.
// rmap (when the screen ran in key order): the row at position i; results are at positions.
__global__ __launch_bounds__(256) void finalize1_first_kernel(int64_t n, int splits, const float* __restrict__ pR,
                                                              const double* __restrict__ pD, const int* __restrict__ pK,
                                                              const double* __restrict__ xn2a, ScreenBound bound,
                                                              const int* __restrict__ rmap,
                                                              int* __restrict__ tmp, float* __restrict__ tmpD,
                                                              int* __restrict__ bcount,
                                                              int32_t* __restrict__ codes, float* __restrict__ dist,
                                                              double* __restrict__ rowD, int* __restrict__ rowK) {
  __shared__ int s_wc[4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const bool valid = i < n;
  const int64_t row = (valid && rmap) ? static_cast<int64_t>(rmap[i]) : i;
  bool fail = false;
  if (valid) fail = !finish_top1(i, row, splits, n, pR, pD, pK, xn2a, bound, codes, dist, rowD, rowK);
  const uint64_t m = __ballot(fail);
  if (lane == 0) s_wc[w] = __popcll(m);
  __syncthreads();
  int woff = 0;
  for (int u = 0; u < w; ++u) woff += s_wc[u];
  if (fail) {
    const int64_t slot = static_cast<int64_t>(blockIdx.x) * 256 + woff + __popcll(m & ((1ull << lane) - 1ull));
    tmp[slot] = static_cast<int>(row);
    if (tmpD) {  // the row's tentative exact distance, rounded up: a bound for the second screen's bands
      double Dt = pD[i];
      for (int sp = 1; sp < splits; ++sp) Dt = fmin(Dt, pD[static_cast<int64_t>(sp) * n + i]);
      tmpD[slot] = f32_up_any(Dt);
    }
  }
  if (threadIdx.x == 0) bcount[blockIdx.x] = s_wc[0] + s_wc[1] + s_wc[2] + s_wc[3];
}

// Exclusive prefix sums of the nb block counts (one block of 1024 threads; each thread sums a
// contiguous run, the runs are scanned in LDS), and their total to *total.
__global__ __launch_bounds__(1024) void scan_counts_kernel(const int* __restrict__ cnt, int64_t nb,
                                                           int* __restrict__ offs, int* __restrict__ total) {
  __shared__ int sh[1024];
  const int t = threadIdx.x;
  const int64_t per = (nb + 1023) / 1024;
  const int64_t b0 = t * per, b1 = b0 + per < nb ? b0 + per : nb;
  int sum = 0;
  for (int64_t b = b0; b < b1; ++b) sum += cnt[b];
  sh[t] = sum;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {  // inclusive Hillis-Steele scan
    const int v = t >= off ? sh[t - off] : 0;
    __syncthreads();
    sh[t] += v;
    __syncthreads();
  }
  int run = t > 0 ? sh[t - 1] : 0;
  for (int64_t b = b0; b < b1; ++b) {
    offs[b] = run;
    run += cnt[b];
  }
  if (t == 1023) *total = sh[1023];
}

// rlist[offs[b] + j] = tmp[256 b + j] for j < cnt[b]: the per-block slices packed in block order.
__global__ __launch_bounds__(256) void compact_list_kernel(const int* __restrict__ tmp, const float* __restrict__ tmpD,
                                                           const int* __restrict__ cnt, const int* __restrict__ offs,
                                                           int* __restrict__ rlist, float* __restrict__ rlistD) {
  const int b = blockIdx.x;
  if (static_cast<int>(threadIdx.x) < cnt[b]) {
    rlist[offs[b] + threadIdx.x] = tmp[static_cast<int64_t>(b) * 256 + threadIdx.x];
    if (tmpD) rlistD[offs[b] + threadIdx.x] = tmpD[static_cast<int64_t>(b) * 256 + threadIdx.x];
  }
}

// Top-1 finalize of a second screen over a row list (rows list[0 .. *list_n), their screen results at
// the list positions): the same merge of the splits and certificate, writing each row's result to its
// own index; rows still uncertain (few) go to the next list.
__global__ __launch_bounds__(256) void finalize1_list_kernel(int splits, int64_t ns, const int* __restrict__ list,
                                                             const int* __restrict__ list_n, const float* __restrict__ pR,
                                                             const double* __restrict__ pD, const int* __restrict__ pK,
                                                             const double* __restrict__ xn2a, ScreenBound bound,
                                                             int* __restrict__ rcount, int* __restrict__ rlist,
                                                             int32_t* __restrict__ codes, float* __restrict__ dist,
                                                             double* __restrict__ rowD, int* __restrict__ rowK) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (static_cast<int64_t>(blockIdx.x) * 256 >= *list_n) return;  // whole block past the list
  const bool valid = i < *list_n;
  const int64_t row = valid ? list[i] : 0;
  bool fail = false;
  if (valid) fail = !finish_top1(i, row, splits, ns, pR, pD, pK, xn2a, bound, codes, dist, rowD, rowK);
  list_append(fail, row, rcount, rlist);
}

// Top-1 rescue.  Blocks take kRB listed rows at a time (rows b * kRB .., b = block, block + grid,
// ...) and stream the codebook once for all of them.  For each codeword and row a fp32 direct-form
// distance d_f = sum_t (x_t - c_t)^2 (fma, t ascending) is a filter: its error is at most ~10u of
// the true distance (u = 2^-24; for fp64 rows x is rounded to fp32 first, which moves sqrt(D) by
// at most u ||x||), so every codeword with D <= D_tent passes d_f <= thr = (1 + 2^-20)
// (sqrt(D_tent) + 2^-22 ||x||)^2 + 2^-120, D_tent being the exact distance of the tentative
// winner.  Codewords that pass are scored exactly in fp64 and merged in (D, k) order.  A
// non-finite threshold lets every codeword through (plain exact search).
// Parts: with gridDim.y = P > 1 and room for every listed row's P partial results in partD / partK
// (count * P <= cap), block (b, p) scans only the p-th of P equal codeword ranges and stores its
// (D, k) minimum per row; rescue1_merge then takes the (D, k) minimum over the parts and emits the
// row.  A few listed rows thus spread over P times as many workgroups (the scan of a long codebook
// is the latency of the whole call otherwise).  Without the room, all blocks form one persistent
// grid over the row batches, each scanning the whole codebook and emitting, as with P = 1.
template <int KS>
__global__ __launch_bounds__(256) void rescue1_kernel(RowSrc src, int top, const void* __restrict__ C, int ct,
                                                      int64_t K, const int* __restrict__ rcount,
                                                      const int* __restrict__ rlist, int32_t* __restrict__ codes,
                                                      float* __restrict__ dist, double* __restrict__ rowD,
                                                      int* __restrict__ rowK, double* __restrict__ partD,
                                                      int* __restrict__ partK, int64_t cap) {
  constexpr int DM = 4 * KS;
  constexpr int kRB = 32 / DM;  // rows per batch: their 32 values live in scalar registers
  constexpr int kU = 4;         // codewords per thread in flight
  __shared__ float sx[kRB][DM];
  __shared__ float sthr[kRB];
  __shared__ int srow[kRB];
  __shared__ double wD[4][kRB];
  __shared__ int wK[4][kRB];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int d = src.d;
  const int count = *rcount;
  const int P = static_cast<int>(gridDim.y);
  const bool parted = P > 1 && static_cast<int64_t>(count) * P <= cap;
  const int64_t kpart = parted ? (K + P - 1) / P : K;
  const int64_t kb = parted ? static_cast<int64_t>(blockIdx.y) * kpart : 0;
  const int64_t ke = (kb + kpart < K) ? kb + kpart : K;
#if CRVQ_DEBUG_RESCUE
  if (blockIdx.x == 0 && threadIdx.x == 0) printf("[rescue] rows %d of %ld, K %ld\n", count, (long)src.n, (long)K);
#endif
  const int nbatch = (count + kRB - 1) / kRB;
  // parted: blocks (x, p) share part p's codeword range; otherwise all blocks are one persistent grid
  const int bstart = parted ? static_cast<int>(blockIdx.x) : static_cast<int>(blockIdx.y * gridDim.x + blockIdx.x);
  const int bstep = parted ? static_cast<int>(gridDim.x) : static_cast<int>(gridDim.x * gridDim.y);
  for (int bt = bstart; bt < nbatch; bt += bstep) {
    const int ns = (count - bt * kRB < kRB) ? count - bt * kRB : kRB;  // rows in this batch
    if (tid < kRB) {
      float thr = -__builtin_inff();  // an empty slot passes nothing
      int row = -1;
      double xd[DM];
      if (tid < ns) {
        row = rlist[bt * kRB + tid];
        load_row_exact<DM>(src, row, true, xd);
        double Dt;
        if (codes) {
          // the tentative code is re-scored only when it indexes the book; otherwise the threshold
          // starts at +inf and every codeword is scored exactly
          const int k0 = codes[row];
          const bool okc = k0 >= 0 && k0 < K;
          float c0[DM];
          load_codeword<DM>(C, ct, okc ? k0 : 0, d, okc, c0);
          Dt = 0.0;
#pragma unroll
          for (int t = 0; t < DM; ++t) {
            if (t < d) {
              const double diff = xd[t] - static_cast<double>(c0[t]);
              Dt = Dt + diff * diff;
            }
          }
          if (!okc) Dt = __builtin_inf();
        } else {
          Dt = rowD[static_cast<int64_t>(row) * top];
        }
        double xn2 = 0.0;
#pragma unroll
        for (int t = 0; t < DM; ++t)
          if (t < d) xn2 = xn2 + xd[t] * xd[t];
        const double rt = sqrt(Dt) + 0x1p-22 * sqrt(xn2);
        const double th = (1.0 + 0x1p-20) * rt * rt + 0x1p-120;
        thr = (th <= 3.0e38) ? static_cast<float>(th) * (1.0f + 0x1p-22f) : __builtin_inff();
      } else {
#pragma unroll
        for (int t = 0; t < DM; ++t) xd[t] = 0.0;
      }
#pragma unroll
      for (int t = 0; t < DM; ++t) sx[tid][t] = static_cast<float>(xd[t]);
      sthr[tid] = thr;
      srow[tid] = row;
    }
    __syncthreads();
    float xr[kRB][DM], th[kRB];  // uniform over the block: held in scalar registers
#pragma unroll
    for (int s = 0; s < kRB; ++s) {
      th[s] = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(sthr[s])));
#pragma unroll
      for (int t = 0; t < DM; ++t) xr[s][t] = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(sx[s][t])));
    }
    double bD[kRB];
    int bK[kRB];
#pragma unroll
    for (int s = 0; s < kRB; ++s) {
      bD[s] = __builtin_inf();
      bK[s] = INT_MAX;
    }
    for (int64_t k0 = kb + tid; k0 < ke; k0 += kU * 256) {
      float c[kU][DM];
#pragma unroll
      for (int u = 0; u < kU; ++u) load_codeword<DM>(C, ct, k0 + u * 256, d, k0 + u * 256 < ke, c[u]);
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t k = k0 + u * 256;
        if (k >= ke) continue;
#pragma unroll
        for (int s = 0; s < kRB; ++s) {
          if (s >= ns) continue;  // uniform
          float df = 0.0f;
#pragma unroll
          for (int t = 0; t < DM; ++t) {
            if (t < d) {
              const float diff = xr[s][t] - c[u][t];
              df = __builtin_fmaf(diff, diff, df);
            }
          }
          if (df <= th[s]) {  // rare: score exactly
            double xe[DM];
            load_row_exact<DM>(src, srow[s], true, xe);
            double D = 0.0;
#pragma unroll
            for (int t = 0; t < DM; ++t) {
              if (t < d) {
                const double diff = xe[t] - static_cast<double>(c[u][t]);
                D = D + diff * diff;
              }
            }
            if (cless(D, static_cast<int>(k), bD[s], bK[s])) {
              bD[s] = D;
              bK[s] = static_cast<int>(k);
            }
          }
        }
      }
    }
    // (D, k) minimum per row: within each wave, then over the four waves in wave order
#pragma unroll
    for (int s = 0; s < kRB; ++s) {
      if (s >= ns) continue;  // uniform
#pragma unroll
      for (int m = 1; m < 64; m <<= 1) {
        const double oD = __shfl_xor(bD[s], m);
        const int oK = __shfl_xor(bK[s], m);
        if (cless(oD, oK, bD[s], bK[s])) {
          bD[s] = oD;
          bK[s] = oK;
        }
      }
      if (lane == 0) {
        wD[w][s] = bD[s];
        wK[w][s] = bK[s];
      }
    }
    __syncthreads();
    if (tid < ns) {
      double D = wD[0][tid];
      int k = wK[0][tid];
      for (int ww = 1; ww < 4; ++ww) {
        if (cless(wD[ww][tid], wK[ww][tid], D, k)) {
          D = wD[ww][tid];
          k = wK[ww][tid];
        }
      }
      if (parted) {
        const int64_t slot = static_cast<int64_t>(bt) * kRB + tid;
        partD[slot * P + blockIdx.y] = D;
        partK[slot * P + blockIdx.y] = k;
      } else {
        const double ED[1] = {D};
        const int EK[1] = {k};
        emit_row<1>(srow[tid], ED, EK, top, 1, codes, dist, rowD, rowK);
      }
    }
    __syncthreads();
  }
}

// The (D, k) minimum over the P parts of every listed row, emitted (parted rescues only).
__global__ __launch_bounds__(256) void rescue1_merge(int top, int P, int64_t cap, const int* __restrict__ rcount,
                                                     const int* __restrict__ rlist, const double* __restrict__ partD,
                                                     const int* __restrict__ partK, int32_t* __restrict__ codes,
                                                     float* __restrict__ dist, double* __restrict__ rowD,
                                                     int* __restrict__ rowK) {
  const int count = *rcount;
  if (!(P > 1 && static_cast<int64_t>(count) * P <= cap)) return;
  for (int64_t slot = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; slot < count;
       slot += static_cast<int64_t>(gridDim.x) * 256) {
    double D = partD[slot * P];
    int k = partK[slot * P];
    for (int q = 1; q < P; ++q) {
      if (cless(partD[slot * P + q], partK[slot * P + q], D, k)) {
        D = partD[slot * P + q];
        k = partK[slot * P + q];
      }
    }
    const double ED[1] = {D};
    const int EK[1] = {k};
    emit_row<1>(rlist[slot], ED, EK, top, 1, codes, dist, rowD, rowK);
  }
}

// Top-1 rescue launch: codebooks of at least kRescuePartMinK codewords are scanned in
// kRescueParts ranges when the free partial-result space (cap entries) holds them.
template <int KS>
hipError_t launch_rescue1(const RowSrc& src, int top, const void* C, int ct, int64_t K, const int* rcount,
                          const int* rlist, int32_t* codes, float* dist, double* rowD, int* rowK, double* partD,
                          int* partK, int64_t cap, hipStream_t stream) {
  constexpr int kRB = 32 / (4 * KS);
  const int P = (K >= kRescuePartMinK && partD && partK) ? kRescueParts : 1;
  int64_t gx = cdiv(src.n, kRB);
  const int64_t gmax = kRescueBlocks / P > 1 ? kRescueBlocks / P : 1;
  if (gx > gmax) gx = gmax;
  hipLaunchKernelGGL((rescue1_kernel<KS>), dim3(static_cast<unsigned>(gx), static_cast<unsigned>(P)), dim3(256), 0,
                     stream, src, top, C, ct, K, rcount, rlist, codes, dist, rowD, rowK, partD, partK, cap);
  if (P > 1)
    hipLaunchKernelGGL(rescue1_merge, dim3(64), dim3(256), 0, stream, top, P, cap, rcount, rlist, partD, partK, codes,
                       dist, rowD, rowK);
  return hipGetLastError();
}

// Exact fp64 search of every listed row over the whole codebook.  Persistent: block b takes rows
// b, b + grid, ... of the list; its 256 threads split the codebook (8 codewords per thread and
// round, all loaded before any is scored) and the per-thread (D, k) lists are merged in LDS.
template <int KS, int NB>
__global__ __launch_bounds__(256) void rescue_kernel(RowSrc src, int top, const void* __restrict__ C, int ct, int64_t K,
                                                     const int* __restrict__ rcount, const int* __restrict__ rlist,
                                                     int32_t* __restrict__ codes, float* __restrict__ dist,
                                                     double* __restrict__ rowD, int* __restrict__ rowK) {
  constexpr int DM = 4 * KS;
  constexpr int kRU = 8;
  __shared__ double sD[128 * NB];
  __shared__ int sK[128 * NB];
  const int tid = threadIdx.x;
  const int d = src.d;
  const int need = static_cast<int>((top < K) ? top : K);
  const int count = *rcount;
  for (int f = blockIdx.x; f < count; f += gridDim.x) {
    const int64_t row = rlist[f];
    double xr[DM];
    load_row_exact<DM>(src, row, true, xr);
    double TD[NB];
    int TK[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      TD[j] = __builtin_inf();
      TK[j] = INT_MAX;
    }
    for (int64_t k0 = tid; k0 < K; k0 += kRU * 256) {
      float cw[kRU][DM];
#pragma unroll
      for (int u = 0; u < kRU; ++u) {
        const int64_t k = k0 + u * 256;
        load_codeword<DM>(C, ct, k, d, k < K, cw[u]);
      }
#pragma unroll
      for (int u = 0; u < kRU; ++u) {
        const int64_t k = k0 + u * 256;
        if (k < K) {
          double acc = 0.0;
#pragma unroll
          for (int t = 0; t < DM; ++t) {
            if (t < d) {
              const double diff = xr[t] - static_cast<double>(cw[u][t]);
              acc = acc + diff * diff;
            }
          }
          list_insert<NB>(TD, TK, acc, static_cast<int>(k));
        }
      }
    }
    for (int stride = 128; stride >= 1; stride >>= 1) {
      if (tid >= stride && tid < 2 * stride) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          sD[(tid - stride) * NB + j] = TD[j];
          sK[(tid - stride) * NB + j] = TK[j];
        }
      }
      __syncthreads();
      if (tid < stride) {
        double OD[NB];
        int OK[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          OD[j] = sD[tid * NB + j];
          OK[j] = sK[tid * NB + j];
        }
        list_merge<NB>(TD, TK, OD, OK);
      }
      __syncthreads();
    }
    if (tid == 0) emit_row<NB>(row, TD, TK, top, need, codes, dist, rowD, rowK);
  }
}

// ------------------------------------------------------------------------------------------------
// beam bookkeeping
// ------------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void beam_merge_kernel(int64_t n, int n_par, int n_next, int beam, int step,
                                                         int n_books, const double* __restrict__ rowD,
                                                         const int* __restrict__ rowK, RowSrc src0,
                                                         const double* __restrict__ res_in,
                                                         double* __restrict__ res_out, const int* __restrict__ tup_in,
                                                         int* __restrict__ tup_out, double* __restrict__ err_out,
                                                         const void* __restrict__ book, int bt, int64_t K, int d) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n) return;
  int head[kMaxBeam];
  for (int b = 0; b < n_par; ++b) head[b] = 0;
  const int64_t off0 = (step == 0) ? row_offset(src0, i) : 0;
  for (int s = 0; s < n_next; ++s) {
    int bb = -1, bk = 0;
    double bD = 0.0;
    for (int b = 0; b < n_par; ++b) {
      if (head[b] >= beam) continue;
      const int64_t r = (i * n_par + b) * beam + head[b];
      const int k = rowK[r];
      if (k < 0 || k >= K) continue;
      const double D = rowD[r];
      if (bb < 0 || D < bD || (D == bD && (b < bb || (b == bb && k < bk)))) {
        bb = b;
        bk = k;
        bD = D;
      }
    }
    double* ro = res_out + (i * n_next + s) * d;
    int* to = tup_out + (i * n_next + s) * n_books;
    if (bb < 0) {  // cannot happen when n_next = min(beam, n_par * K); kept as a guard
      err_out[i * n_next + s] = __builtin_inf();
      for (int t = 0; t < d; ++t) ro[t] = 0.0;
      for (int u = 0; u <= step; ++u) to[u] = 0;
      continue;
    }
    head[bb] += 1;
    for (int t = 0; t < d; ++t) {
      const double parent = (step == 0) ? row_elem(src0, off0, t) : res_in[(i * n_par + bb) * d + t];
      ro[t] = parent - cb_elem(book, bt, bk, d, t);
    }
    for (int u = 0; u < step; ++u) to[u] = tup_in[(i * n_par + bb) * n_books + u];
    to[step] = bk;
    err_out[i * n_next + s] = bD;
  }
}

// The same selection with one wave per vector: the n_par x beam candidates (up to 4 per lane) are
// ranked by counting, for each, the candidates with a smaller key (D, parent, code); a candidate
// of rank r < n_next writes child slot r.  Keys are distinct (a parent lists a codeword once;
// invalid entries get +inf and a key past every parent), so the ranks are a permutation and the
// children come out in the order of the sequential merge above.
__global__ __launch_bounds__(256) void beam_merge_wave(int64_t n, int n_par, int n_next, int beam, int step,
                                                       int n_books, const double* __restrict__ rowD,
                                                       const int* __restrict__ rowK, RowSrc src0,
                                                       const double* __restrict__ res_in, double* __restrict__ res_out,
                                                       const int* __restrict__ tup_in, int* __restrict__ tup_out,
                                                       double* __restrict__ err_out, const void* __restrict__ book,
                                                       int bt, int64_t K, int d) {
  const int lane = threadIdx.x & 63;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (i >= n) return;  // whole waves leave together; no barriers below
  const int nc = n_par * beam;  // <= kMaxBeam * kMaxBeam = 256
  double cD[4];
  int cB[4], cK[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = lane + 64 * q;
    cD[q] = __builtin_inf();
    cB[q] = n_par + c;  // invalid: after every parent, distinct
    cK[q] = -1;
    if (c < nc) {
      const int b = c / beam;
      const int64_t r = (i * n_par + b) * beam + (c - b * beam);
      const int k = rowK[r];
      if (k >= 0 && k < K) {
        cD[q] = rowD[r];
        cB[q] = b;
        cK[q] = k;
      }
    }
  }
  auto less = [](double Da, int ba, int ka, double Db, int bb, int kb) {
    return Da < Db || (Da == Db && (ba < bb || (ba == bb && ka < kb)));
  };
  int rank[4] = {0, 0, 0, 0};
  const int rounds = (nc + 63) / 64;  // candidate slots in use per lane (uniform)
  for (int q2 = 0; q2 < rounds; ++q2) {
    const int jn = (nc - 64 * q2 < 64) ? nc - 64 * q2 : 64;
    for (int j = 0; j < jn; ++j) {
      const double oD = __shfl(cD[q2], j);
      const int oB = __shfl(cB[q2], j);
      const int oK = __shfl(cK[q2], j);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q < rounds) rank[q] += less(oD, oB, oK, cD[q], cB[q], cK[q]) ? 1 : 0;
    }
  }
  const int64_t off0 = (step == 0) ? row_offset(src0, i) : 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = lane + 64 * q;
    if (c >= nc || rank[q] >= n_next) continue;
    const int s = rank[q];
    double* ro = res_out + (i * n_next + s) * d;
    int* to = tup_out + (i * n_next + s) * n_books;
    if (cK[q] < 0) {  // cannot happen when n_next = min(beam, n_par * K); kept as a guard
      err_out[i * n_next + s] = __builtin_inf();
      for (int t = 0; t < d; ++t) ro[t] = 0.0;
      for (int u = 0; u <= step; ++u) to[u] = 0;
      continue;
    }
    const int b = cB[q];
    if (d == 8 && step > 0 && bt == ET_F32 && (reinterpret_cast<uintptr_t>(book) & 15) == 0) {  // 16-byte accesses
      const double2* pr = reinterpret_cast<const double2*>(res_in + (i * n_par + b) * 8);
      const float4* cw = reinterpret_cast<const float4*>(static_cast<const float*>(book) + static_cast<int64_t>(cK[q]) * 8);
      const float4 c0 = cw[0], c1 = cw[1];
      const float cc[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
      double2* rw = reinterpret_cast<double2*>(ro);
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const double2 pv = pr[h];
        rw[h] = make_double2(pv.x - static_cast<double>(cc[2 * h]), pv.y - static_cast<double>(cc[2 * h + 1]));
      }
    } else {
      for (int t = 0; t < d; ++t) {
        const double parent = (step == 0) ? row_elem(src0, off0, t) : res_in[(i * n_par + b) * d + t];
        ro[t] = parent - cb_elem(book, bt, cK[q], d, t);
      }
    }
    for (int u = 0; u < step; ++u) to[u] = tup_in[(i * n_par + b) * n_books + u];
    to[step] = cK[q];
    err_out[i * n_next + s] = cD[q];
  }
}

// The same selection with eight lanes per vector (n_par <= 8, beam <= 8): lane b holds parent b's
// child list, which the search emits in (D, code) order; at every step the eight list heads are
// reduced to the smallest key (D, parent, code) with xor shuffles inside the lane group, the winning
// parent drops its head, and lane s keeps the winner of step s and writes child slot s.  Exhausted or
// invalid heads carry +inf and a parent index past every parent (distinct per lane), so the winners
// come out in the order of the sequential merge above.
__global__ __launch_bounds__(256) void beam_merge_lanes(int64_t n, int n_par, int n_next, int beam, int step,
                                                        int n_books, const double* __restrict__ rowD,
                                                        const int* __restrict__ rowK, RowSrc src0,
                                                        const double* __restrict__ res_in, double* __restrict__ res_out,
                                                        const int* __restrict__ tup_in, int* __restrict__ tup_out,
                                                        double* __restrict__ err_out, const void* __restrict__ book,
                                                        int bt, int64_t K, int d) {
  const int sub = threadIdx.x & 7;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 32 + (threadIdx.x >> 3);
  const bool live = i < n;  // no early exit: the lane groups shuffle among themselves only
  const bool has = live && sub < n_par;
  double hD[8];
  int hK[8];
#pragma unroll
  for (int h = 0; h < 8; ++h) {
    hD[h] = __builtin_inf();
    hK[h] = -1;
    if (has && h < beam) {
      const int64_t r = (i * n_par + sub) * beam + h;
      const int k = rowK[r];
      if (k >= 0 && k < K) {
        hD[h] = rowD[r];
        hK[h] = k;
      }
    }
  }
  auto less = [](double Da, int ba, int ka, double Db, int bb, int kb) {
    return Da < Db || (Da == Db && (ba < bb || (ba == bb && ka < kb)));
  };
  double myD = __builtin_inf();
  int myB = -1, myK = -1;
  for (int s = 0; s < n_next; ++s) {
    const bool valid_head = hK[0] >= 0;
    double mD = valid_head ? hD[0] : __builtin_inf();
    int mB = valid_head ? sub : n_par + sub;
    int mK = hK[0];
#pragma unroll
    for (int m = 1; m < 8; m <<= 1) {
      const double oD = __shfl_xor(mD, m);
      const int oB = __shfl_xor(mB, m);
      const int oK = __shfl_xor(mK, m);
      if (less(oD, oB, oK, mD, mB, mK)) {
        mD = oD;
        mB = oB;
        mK = oK;
      }
    }
    if (s == sub) {
      myD = mD;
      myB = mB;
      myK = mK;
    }
    if (valid_head && mB == sub) {  // this parent's head was taken: drop it
#pragma unroll
      for (int h = 0; h < 7; ++h) {
        hD[h] = hD[h + 1];
        hK[h] = hK[h + 1];
      }
      hD[7] = __builtin_inf();
      hK[7] = -1;
    }
  }
  if (!live || sub >= n_next) return;
  const int s = sub;
  double* ro = res_out + (i * n_next + s) * d;
  int* to = tup_out + (i * n_next + s) * n_books;
  if (myK < 0 || myB >= n_par) {  // cannot happen when n_next = min(beam, n_par * K); kept as a guard
    err_out[i * n_next + s] = __builtin_inf();
    for (int t = 0; t < d; ++t) ro[t] = 0.0;
    for (int u = 0; u <= step; ++u) to[u] = 0;
    return;
  }
  if (d == 8 && step > 0 && bt == ET_F32 && (reinterpret_cast<uintptr_t>(book) & 15) == 0) {  // 16-byte accesses
    const double2* pr = reinterpret_cast<const double2*>(res_in + (i * n_par + myB) * 8);
    const float4* cw = reinterpret_cast<const float4*>(static_cast<const float*>(book) + static_cast<int64_t>(myK) * 8);
    const float4 c0 = cw[0], c1 = cw[1];
    const float cc[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
    double2* rw = reinterpret_cast<double2*>(ro);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const double2 pv = pr[h];
      rw[h] = make_double2(pv.x - static_cast<double>(cc[2 * h]), pv.y - static_cast<double>(cc[2 * h + 1]));
    }
  } else {
    const int64_t off0 = (step == 0) ? row_offset(src0, i) : 0;
    for (int t = 0; t < d; ++t) {
      const double parent = (step == 0) ? row_elem(src0, off0, t) : res_in[(i * n_par + myB) * d + t];
      ro[t] = parent - cb_elem(book, bt, myK, d, t);
    }
  }
  for (int u = 0; u < step; ++u) to[u] = tup_in[(i * n_par + myB) * n_books + u];
  to[step] = myK;
  err_out[i * n_next + s] = myD;
}

__global__ __launch_bounds__(256) void beam_emit_kernel(int64_t n, int64_t vpr, int n_par, int n_books,
                                                        const int* __restrict__ tup, const double* __restrict__ err,
                                                        CodePtrs outs, float* __restrict__ err_out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t r = i / vpr;
  const int64_t g = i - r * vpr;
  for (int t = 0; t < n_books; ++t) outs.q[t][r * outs.ld[t] + g] = tup[(i * n_par) * n_books + t];
  if (err_out) err_out[i] = static_cast<float>(err[i * n_par]);
}

template <class OPS, int NB, int CB, int NC = 1>
hipError_t launch_screen_t(const RowSrc& src, const void* C, int ct, int64_t K, const ScreenPlan& p,
                           const ScreenWs& w, hipStream_t stream) {
  dim3 grid(static_cast<unsigned>(p.grid_x), static_cast<unsigned>(p.splits));
  hipLaunchKernelGGL((screen_kernel<OPS, NB, CB, NC>), grid, dim3(256), 0, stream, src, w.apack, w.cnp, p.tiles,
                     p.tiles_per_split, C, ct, K, w.pT, w.pM, w.pR, w.pD, w.pK, w.xn2);
  return hipGetLastError();
}

template <class OPS>
hipError_t launch_screen_ops(const RowSrc& src, const void* C, int ct, int64_t K, const ScreenPlan& p,
                             const ScreenWs& w, hipStream_t stream) {
  switch (p.nb) {
    case 1:
      if (p.chunk > 1)
        return p.cb == CRVQ_CB_WIDE ? launch_screen_t<OPS, 1, CRVQ_CB_WIDE, CRVQ_CHUNK>(src, C, ct, K, p, w, stream)
                                    : launch_screen_t<OPS, 1, 2, CRVQ_CHUNK>(src, C, ct, K, p, w, stream);
      return p.cb == CRVQ_CB_WIDE ? launch_screen_t<OPS, 1, CRVQ_CB_WIDE>(src, C, ct, K, p, w, stream)
                                  : launch_screen_t<OPS, 1, 2>(src, C, ct, K, p, w, stream);
    case 2:
      if (p.chunk > 1)
        return p.cb == CRVQ_CB_WIDE ? launch_screen_t<OPS, 2, CRVQ_CB_WIDE, CRVQ_CHUNK_TOPB>(src, C, ct, K, p, w, stream)
                                    : launch_screen_t<OPS, 2, 2, CRVQ_CHUNK_TOPB>(src, C, ct, K, p, w, stream);
      return p.cb == CRVQ_CB_WIDE ? launch_screen_t<OPS, 2, CRVQ_CB_WIDE>(src, C, ct, K, p, w, stream)
                                  : launch_screen_t<OPS, 2, 2>(src, C, ct, K, p, w, stream);
    case 4:
      if (p.chunk > 1) return launch_screen_t<OPS, 4, 4, CRVQ_CHUNK_TOPB>(src, C, ct, K, p, w, stream);
      return launch_screen_t<OPS, 4, 4>(src, C, ct, K, p, w, stream);
    case 8:
      if (p.chunk > 1) return launch_screen_t<OPS, 8, 2, CRVQ_CHUNK_TOPB>(src, C, ct, K, p, w, stream);
      return launch_screen_t<OPS, 8, 2>(src, C, ct, K, p, w, stream);
    case 16: return launch_screen_t<OPS, 16, 1>(src, C, ct, K, p, w, stream);
  }
  return hipErrorInvalidValue;
}

template <int KS, int NB>
hipError_t launch_finalize_t(const RowSrc& src, const void* C, int ct, int64_t K, int top, const ScreenPlan& p,
                             const ScreenWs& w, const ScreenBound& bound, int32_t* codes, float* dist, double* rowD,
                             int* rowK, hipStream_t stream) {
  hipLaunchKernelGGL((finalize_kernel<KS, NB>), dim3(static_cast<unsigned>(cdiv(src.n, 256))), dim3(256), 0, stream,
                     src, p.splits, NB > 1 ? static_cast<int>(p.chunk) : 1, p.tiles_per_split, p.tiles, top, w.pT,
                     w.pM, w.pR, w.pD, w.pK, w.xn2, C, ct, K, bound, w.rcount, w.rlist, codes,
                     dist, rowD, rowK);
  const int64_t rgrid = src.n < kRescueBlocks ? src.n : kRescueBlocks;
  if (NB == 1 && CRVQ_RESCUE_FILTER)  // pD / pK are free once the finalize has read them
    return launch_rescue1<KS>(src, top, C, ct, K, w.rcount, w.rlist, codes, dist, rowD, rowK, w.pD, w.pK,
                              static_cast<int64_t>(p.splits) * src.n, stream);
  else
    hipLaunchKernelGGL((rescue_kernel<KS, NB>), dim3(static_cast<unsigned>(rgrid)), dim3(256), 0, stream, src, top, C,
                       ct, K, w.rcount, w.rlist, codes, dist, rowD, rowK);
  return hipGetLastError();
}

template <int KS>
hipError_t launch_finalize_ks(const RowSrc& src, const void* C, int ct, int64_t K, int top, const ScreenPlan& p,
                              const ScreenWs& w, const ScreenBound& bound, int32_t* codes, float* dist, double* rowD,
                              int* rowK, hipStream_t stream) {
  switch (p.nb) {
    case 1: return launch_finalize_t<KS, 1>(src, C, ct, K, top, p, w, bound, codes, dist, rowD, rowK, stream);
    case 2: return launch_finalize_t<KS, 2>(src, C, ct, K, top, p, w, bound, codes, dist, rowD, rowK, stream);
    case 4: return launch_finalize_t<KS, 4>(src, C, ct, K, top, p, w, bound, codes, dist, rowD, rowK, stream);
    case 8: return launch_finalize_t<KS, 8>(src, C, ct, K, top, p, w, bound, codes, dist, rowD, rowK, stream);
    case 16: return launch_finalize_t<KS, 16>(src, C, ct, K, top, p, w, bound, codes, dist, rowD, rowK, stream);
  }
  return hipErrorInvalidValue;
}

// bf16 rows against a bf16 codebook: the 32 x 32 screen runs one MFMA per tile on exact operands.
bool s32_exact_operands(int x_type, int ct) { return x_type == ET_BF16 && ct == ET_BF16; }

// The certification bound of a screen mode.  fp32 MFMA: the accumulation and ||c||^2 roundings.
// Split bf16: a wider accumulation allowance (the 32-term bf16 MFMA sum, measured well below it),
// the split remainder 2^-15 ||x|| R for each operand that is not bf16 already, and an absolute
// term for subnormal operands or partial sums that the matrix core may flush.
ScreenBound screen_bound(const ScreenPlan& p, int x_type, int ct, int d, const float* alpha, bool one_mfma = false) {
  ScreenBound b;
  b.acc_ulps = static_cast<double>(4 * d + 24);
  b.split_coef = 0.0;
  b.abs_coef = 0.0;
  b.alpha = nullptr;
  b.row_e = nullptr;
  if (p.s32) {
    // remainders of both splits and the dropped c2.x2, each <= 2^-22 sum |c_t| |2 x_t|; none when
    // both operands are bf16 (exact in fp16 under the scale)
    // one MFMA per tile on fp16-rounded operands instead: the dropped c1.x2 + c2.x1 + c2.x2 with
    // |x2| <= 2^-11 |x1|, |c2| <= 2^-11 |c1| is at most 2^-10 (1 + 2^-10) sum |c_t| |2 x_t| <= 2^-9 (1 + 2^-10) ||x|| R
    if (!s32_exact_operands(x_type, ct)) b.split_coef = one_mfma ? 0x1p-9 * (1.0 + 0x1p-9) : 0x1p-19;
    b.alpha = alpha;
  } else if (p.split) {
    if (b.acc_ulps < 96.0) b.acc_ulps = 96.0;
    const int inexact = (x_type != ET_BF16 ? 1 : 0) + (ct != ET_BF16 ? 1 : 0);
    b.split_coef = 0x1p-15 * static_cast<double>(inexact) * (1.0 + 0x1p-6);
    b.abs_coef = 0x1p-118;
  }
  return b;
}

}  // namespace

static int next_pow2_nb(int top) {
  int nb = 1;
  while (nb < top) nb <<= 1;
  return nb;
}

ScreenPlan plan_screen(int64_t n_rows, int d, int64_t K, int top) {
  ScreenPlan p;
  // CRVQ_MIN_TRACKED_TILES = 2 would make the exact rescue almost never needed, but its extra VALU
  // work and registers cost more screen time (12 % at K = 65536) than the rescues it saves.
  p.nb = next_pow2_nb(top < CRVQ_MIN_TRACKED_TILES ? CRVQ_MIN_TRACKED_TILES : top);
  p.cb = p.nb <= 2 ? CRVQ_CB_WIDE : (p.nb == 4 ? 4 : (p.nb == 8 ? 2 : 1));
  // d <= 8: one split-bf16 MFMA per tile (a quarter of the matrix-core time of the two fp32 steps)
  p.split = (CRVQ_SPLIT_SCREEN && d <= 8) ? 1 : 0;
  p.ks = p.split ? 2 : (d <= 4 ? 1 : (d <= 8 ? 2 : 4));
  p.tiles = cdiv(K, 16);
  p.grid_x = cdiv(n_rows, 64 * p.cb);
  int64_t splits = 1;
  const int64_t want_blocks = 2048;
  if (p.grid_x < want_blocks) {
    int64_t want = cdiv(want_blocks, p.grid_x > 0 ? p.grid_x : 1);
    int64_t maxs = p.tiles / 32 > 1 ? p.tiles / 32 : 1;
    splits = want < maxs ? want : maxs;
  }
  // small codebooks cannot be split further: spread the rows over more, smaller workgroups instead
  if (p.grid_x * splits < 1024 && p.nb <= 2) {
    p.cb = 2;
    p.grid_x = cdiv(n_rows, 64 * p.cb);
  }
  p.tiles_per_split = cdiv(p.tiles, splits);
  p.splits = static_cast<int>(cdiv(p.tiles, p.tiles_per_split));
  p.chunk = (p.tiles_per_split >= CRVQ_CHUNK_MIN_TILES && p.nb <= 8) ? (p.nb == 1 ? CRVQ_CHUNK : CRVQ_CHUNK_TOPB) : 1;
  // Long top-1 searches: 32 x 32 split-fp16 tiles (two MFMAs per 1024 values instead of four).
  // The same rows per workgroup and codebook splits, counted in 32-codeword tiles.
  p.s32 = (p.split && CRVQ_S32_SCREEN && p.nb == 1 && p.tiles_per_split >= CRVQ_S32_MIN_TILES) ? 1 : 0;
  p.prune = 0;
  if (p.s32) {
    p.cb = CRVQ_S32_CB;
    p.grid_x = cdiv(n_rows, 128 * p.cb);
    p.tiles = cdiv(K, kS32Tile);
    // many rows: codebook and rows in key order, chunks of two tiles skipped when certified useless
    // (only without codebook splits: a split would see a slice of the key order and prune little)
    p.prune = (CRVQ_PRUNE && CRVQ_S32_CHUNK == 2 && splits == 1 && n_rows >= kPruneMinRows) ? 1 : 0;
    if (p.prune) p.tiles += p.tiles & 1;  // whole chunks; a padding tile never wins
    p.tiles_per_split = cdiv(p.tiles, splits);
    if (p.prune) p.tiles_per_split += p.tiles_per_split & 1;
    p.splits = static_cast<int>(cdiv(p.tiles, p.tiles_per_split));
    p.chunk = CRVQ_S32_CHUNK;
  }
  return p;
}

ScreenWs carve_screen(WsCursor& ws, const ScreenPlan& p, int64_t n_rows, int64_t K_alloc) {
  ScreenWs w;
  const int64_t tiles = cdiv(K_alloc, 16);
  w.corder = w.ckey = w.coff = w.hist = w.rkey = w.rord = nullptr;
  w.cbnd = nullptr;
  w.cbnd3 = nullptr;
  w.cminS = w.cmaxP = nullptr;
  w.prm = nullptr;
  w.tD = w.lD = nullptr;
  w.xe = nullptr;
  if (p.s32) {
    // 32-codeword tiles of 768 fp16, the scale reduction's partial maxima and alpha
    const int64_t t32 = p.tiles > cdiv(K_alloc, kS32Tile) ? p.tiles : cdiv(K_alloc, kS32Tile);
    w.apack = ws.take<float>(static_cast<size_t>(t32 * kS32TileHalves / 2));
    w.cnp = nullptr;
    w.smax = ws.take<float>(static_cast<size_t>(kS32MaxParts + 1));
    if (p.prune) {
      const int64_t nch = t32 / 2 + 1;
      w.corder = ws.take<int>(static_cast<size_t>(t32 * kS32Tile));
      w.ckey = ws.take<int>(static_cast<size_t>(K_alloc));
      w.coff = ws.take<int>(static_cast<size_t>(kPruneKeys));
      // key counts, the fine histograms and their lookup table (3 x kPruneFine bytes)
      w.hist = ws.take<int>(static_cast<size_t>(2 * kPruneKeys + 3 * kPruneFine + 3 * kPruneFine / 4));
      w.cbnd = ws.take<uint4>(static_cast<size_t>(nch));
      w.cbnd3 = ws.take<uint2>(static_cast<size_t>(nch));
      w.cminS = ws.take<uint32_t>(static_cast<size_t>(nch));
      w.cmaxP = ws.take<uint32_t>(static_cast<size_t>(nch));
      w.prm = ws.take<float>(8 + 5 * kPruneParts);  // the parameters, then the partial ranges
      w.rkey = ws.take<int>(static_cast<size_t>(n_rows));
      w.rord = ws.take<int>(static_cast<size_t>(n_rows));
      w.tD = ws.take<float>(static_cast<size_t>(cdiv(n_rows, 256) * 256));
      w.lD = ws.take<float>(static_cast<size_t>(n_rows));
    }
  } else {
    // fp32: 64 lanes x ks floats per tile; split: 16 codewords x 16 bf16 per tile
    w.apack = ws.take<float>(static_cast<size_t>(p.split ? tiles * 128 : tiles * 64 * p.ks));
    w.cnp = ws.take<float>(static_cast<size_t>(tiles * 16));
    w.smax = nullptr;
  }
  w.pR = ws.take<float>(static_cast<size_t>(p.splits) * n_rows);
  w.rcount = ws.take<int>(2);
  w.rlist = ws.take<int>(static_cast<size_t>(n_rows));
  w.rlist2 = p.s32 ? ws.take<int>(static_cast<size_t>(cdiv(n_rows, 256) * 256)) : nullptr;
  w.bcount = p.s32 ? ws.take<int>(static_cast<size_t>(2 * cdiv(n_rows, 256))) : nullptr;
  if (p.nb == 1) {
    w.pT = nullptr;
    w.pM = nullptr;
    w.pD = ws.take<double>(static_cast<size_t>(p.splits) * n_rows);
    w.pK = ws.take<int>(static_cast<size_t>(p.splits) * n_rows);
    w.xn2 = ws.take<double>(static_cast<size_t>(n_rows));
    w.xe = p.s32 ? ws.take<float>(static_cast<size_t>(n_rows)) : nullptr;
  } else {
    w.pT = ws.take<int>(static_cast<size_t>(p.splits) * 4 * p.nb * n_rows);
    w.pM = ws.take<float>(static_cast<size_t>(p.splits) * 4 * p.nb * n_rows);
    w.pD = nullptr;
    w.pK = nullptr;
    w.xn2 = nullptr;
  }
  return w;
}

hipError_t launch_screen(const RowSrc& src, const void* C, int ct, int64_t K, int top, const ScreenPlan& p,
                         const ScreenWs& w, int32_t* out_codes, float* out_dist, double* rowD, int* rowK,
                         hipStream_t stream) {
  if (src.n <= 0) return hipSuccess;
  hipError_t e;
  if (p.s32) {
    const int64_t count = K * src.d;
    int nparts = static_cast<int>(cdiv(count, 4096));
    if (nparts > kS32MaxParts) nparts = kS32MaxParts;
    if (nparts < 1) nparts = 1;
    float* alpha = w.smax + kS32MaxParts;
    uint16_t* ap = reinterpret_cast<uint16_t*>(w.apack);
    hipLaunchKernelGGL(cb_absmax_partial, dim3(nparts), dim3(256), 0, stream, C, ct, count, w.smax);
    PruneData pd = {};
    const int jp = 0;                    // the coordinate of the second band
    const int jq = src.d > 1 ? 1 : 0;    // and of the third
    if (p.prune) {
      // the codebook in key order (the packed tiles follow it), its chunk ranges, then the rows
      RowSrc cbs;
      cbs.base = C;
      cbs.type = ct;
      cbs.d = src.d;
      cbs.vpr = 1;
      cbs.ld = src.d;
      cbs.n = K;
      const int64_t nch = p.tiles / 2;
      const int sparts = static_cast<int>(cdiv(K, 256) < kPruneParts ? cdiv(K, 256) : kPruneParts);
      hipLaunchKernelGGL(prune_stats_partial, dim3(sparts), dim3(256), 0, stream, C, ct, K, src.d, jp, jq, w.prm + 8,
                         w.hist);
      int* fine = w.hist + 2 * kPruneKeys;
      hipLaunchKernelGGL((prune_fine_kernel<kPruneCbThreads>), dim3(static_cast<unsigned>(cdiv(K, kPruneTile))),
                         dim3(kPruneCbThreads), 0, stream, cbs,
                         jp, jq, w.prm + 8, sparts, w.prm, fine);
      uint8_t* lut = reinterpret_cast<uint8_t*>(fine + 3 * kPruneFine);
      hipLaunchKernelGGL(prune_lut_kernel, dim3(1), dim3(256), 0, stream, fine, lut);
      hipLaunchKernelGGL((prune_count_kernel<kPruneCbThreads, kPruneCbTile>),
                         dim3(static_cast<unsigned>(cdiv(K, kPruneCbTile))), dim3(kPruneCbThreads), 0, stream, cbs,
                         jp, jq, w.prm + 8, sparts, w.prm, lut, w.ckey, w.hist);
      hipLaunchKernelGGL(prune_scan_kernel, dim3(1), dim3(1024), 0, stream, w.hist, w.coff);
      hipLaunchKernelGGL(prune_fill_kernel, dim3(static_cast<unsigned>(cdiv(p.tiles * kS32Tile, 256))), dim3(256), 0,
                         stream, w.corder, p.tiles * kS32Tile, -1);
      hipLaunchKernelGGL((prune_order_kernel<kPruneCbThreads, kPruneCbTile>),
                         dim3(static_cast<unsigned>(cdiv(K, kPruneCbTile))), dim3(kPruneCbThreads), 0, stream,
                         w.ckey, K, w.hist, w.corder);
      hipLaunchKernelGGL(prep_codebook_s32, dim3(static_cast<unsigned>(cdiv(p.tiles * kS32Tile, 256))), dim3(256), 0,
                         stream, C, ct, K, src.d, p.tiles, w.smax, nparts, w.corder, ap, alpha, w.rcount);
      hipLaunchKernelGGL(prune_chunks_kernel, dim3(static_cast<unsigned>(cdiv(nch, 4))), dim3(256), 0, stream, C, ct,
                         K, src.d, jp, jq, w.corder, alpha, nch, w.cbnd, w.cbnd3);
      hipLaunchKernelGGL(prune_envelope_kernel, dim3(1), dim3(1024), 0, stream, w.cbnd, static_cast<int>(nch), w.cminS,
                         w.cmaxP, w.prm);
      hipLaunchKernelGGL((prune_count_kernel<kPruneRowThreads, kPruneRowTile>),
                         dim3(static_cast<unsigned>(cdiv(src.n, kPruneRowTile))), dim3(kPruneRowThreads), 0, stream,
                         src, jp, jq, w.prm + 8, sparts, w.prm, lut, w.rkey, w.hist + kPruneKeys);
      hipLaunchKernelGGL(prune_scan_kernel, dim3(1), dim3(1024), 0, stream, w.hist + kPruneKeys, nullptr);
      hipLaunchKernelGGL((prune_order_kernel<kPruneRowThreads, kPruneRowTile>),
                         dim3(static_cast<unsigned>(cdiv(src.n, kPruneRowTile))), dim3(kPruneRowThreads), 0, stream,
                         w.rkey, src.n, w.hist + kPruneKeys, w.rord);
      pd.corder = w.corder;
      pd.coff = w.coff;
      pd.cbnd = w.cbnd;
      pd.cbnd3 = w.cbnd3;
      pd.cminS = w.cminS;
      pd.cmaxP = w.cmaxP;
      pd.rord = w.rord;
      pd.rkey = w.rkey;
      pd.prm = w.prm;
      pd.jp = jp;
      pd.jq = jq;
    } else {
      hipLaunchKernelGGL(prep_codebook_s32, dim3(static_cast<unsigned>(cdiv(p.tiles * kS32Tile, 256))), dim3(256), 0,
                         stream, C, ct, K, src.d, p.tiles, w.smax, nparts, nullptr, ap, alpha, w.rcount);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    dim3 grid(static_cast<unsigned>(p.grid_x), static_cast<unsigned>(p.splits));
    const bool exact = s32_exact_operands(src.type, ct);
    // First screen: one MFMA per tile.  Exact for bf16 rows against a bf16 book; otherwise on
    // fp16-rounded operands, certified with the wider bound.
    // (fp16-rounded operands: each row's own split term, from the screen, replaces the worst case)
    ScreenBound b1 = screen_bound(p, src.type, ct, src.d, alpha, !exact);
    float* const xe = exact ? nullptr : w.xe;
    b1.row_e = xe;
    if (p.prune)
      hipLaunchKernelGGL((screen32_kernel<CRVQ_S32_CB, CRVQ_S32_CHUNK, true, false, false, true>), grid, dim3(256), 0,
                         stream, src, ap, alpha, p.tiles, p.tiles_per_split, C, ct, K, w.pR, w.pD, w.pK, w.xn2, xe,
                         nullptr, nullptr, pd.corder, pd, b1.acc_ulps, b1.split_coef);
    else
      hipLaunchKernelGGL((screen32_kernel<CRVQ_S32_CB, CRVQ_S32_CHUNK, true, false>), grid, dim3(256), 0, stream, src,
                         ap, alpha, p.tiles, p.tiles_per_split, C, ct, K, w.pR, w.pD, w.pK, w.xn2, xe, nullptr, nullptr,
                         nullptr, pd, 0.0, 0.0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (exact && !p.prune) {
      const ScreenBound bound = screen_bound(p, src.type, ct, src.d, alpha);
      return launch_finalize_ks<2>(src, C, ct, K, top, p, w, bound, out_codes, out_dist, rowD, rowK, stream);
    }
    if (exact) {
      // results at key-order positions: certify by position, compact the uncertain rows, rescue them
      const int64_t nbx = cdiv(src.n, 256);
      hipLaunchKernelGGL(finalize1_first_kernel, dim3(static_cast<unsigned>(nbx)), dim3(256), 0, stream, src.n,
                         p.splits, w.pR, w.pD, w.pK, w.xn2, b1, w.rord, w.rlist2, nullptr, w.bcount, out_codes, out_dist,
                         rowD, rowK);
      hipLaunchKernelGGL(scan_counts_kernel, dim3(1), dim3(1024), 0, stream, w.bcount, nbx, w.bcount + nbx, w.rcount);
      hipLaunchKernelGGL(compact_list_kernel, dim3(static_cast<unsigned>(nbx)), dim3(256), 0, stream, w.rlist2, nullptr,
                         w.bcount, w.bcount + nbx, w.rlist, nullptr);
      return launch_rescue1<2>(src, top, C, ct, K, w.rcount, w.rlist, out_codes, out_dist, rowD, rowK, w.pD, w.pK,
                               static_cast<int64_t>(p.splits) * src.n, stream);
    }
    const int64_t nb = cdiv(src.n, 256);
    // the uncertain rows, compacted through rlist2 (free until the second finalize) in row order
    hipLaunchKernelGGL(finalize1_first_kernel, dim3(static_cast<unsigned>(nb)), dim3(256), 0, stream, src.n, p.splits,
                       w.pR, w.pD, w.pK, w.xn2, b1, p.prune ? w.rord : nullptr, w.rlist2, p.prune ? w.tD : nullptr,
                       w.bcount, out_codes, out_dist, rowD, rowK);
    hipLaunchKernelGGL(scan_counts_kernel, dim3(1), dim3(1024), 0, stream, w.bcount, nb, w.bcount + nb, w.rcount);
    hipLaunchKernelGGL(compact_list_kernel, dim3(static_cast<unsigned>(nb)), dim3(256), 0, stream, w.rlist2,
                       p.prune ? w.tD : nullptr, w.bcount, w.bcount + nb, w.rlist, p.prune ? w.lD : nullptr);
    // Second screen, split form (two MFMAs per tile, the tight bound), over the rows the first one
    // left uncertain; what still fails goes to the exact rescue.
    // The listed rows are typically 7-9 % of n: below a few million rows the four waves of a block
    // share 128 of them and split the codebook, above that every wave takes rows of its own.
    // After a pruned first screen the listed rows are in key order with exact distance bounds, and
    // the second screen skips the chunks outside their bands.
    PruneData pd2 = pd;
    pd2.lD = w.lD;
    const bool prune2 = p.prune && CRVQ_PRUNE2;
    if (src.n < kS32SharedRowsMaxN) {
      const dim3 grid2(static_cast<unsigned>(cdiv(src.n, 32 * CRVQ_S32_CB)), static_cast<unsigned>(p.splits));
      if (prune2)
        hipLaunchKernelGGL((screen32_kernel<CRVQ_S32_CB, CRVQ_S32_CHUNK, false, true, true, true>), grid2, dim3(256), 0,
                           stream, src, ap, alpha, p.tiles, p.tiles_per_split, C, ct, K, w.pR, w.pD, w.pK, w.xn2,
                           nullptr, w.rlist, w.rcount, pd.corder, pd2, 0.0, 0.0);
      else
        hipLaunchKernelGGL((screen32_kernel<CRVQ_S32_CB, CRVQ_S32_CHUNK, false, true, true>), grid2, dim3(256), 0,
                           stream, src, ap, alpha, p.tiles, p.tiles_per_split, C, ct, K, w.pR, w.pD, w.pK, w.xn2,
                           nullptr, w.rlist, w.rcount, pd.corder, PruneData{}, 0.0, 0.0);
    } else {
      if (prune2)
        hipLaunchKernelGGL((screen32_kernel<CRVQ_S32_CB, CRVQ_S32_CHUNK, false, true, false, true>), grid, dim3(256), 0,
                           stream, src, ap, alpha, p.tiles, p.tiles_per_split, C, ct, K, w.pR, w.pD, w.pK, w.xn2,
                           nullptr, w.rlist, w.rcount, pd.corder, pd2, 0.0, 0.0);
      else
        hipLaunchKernelGGL((screen32_kernel<CRVQ_S32_CB, CRVQ_S32_CHUNK, false, true, false>), grid, dim3(256), 0,
                           stream, src, ap, alpha, p.tiles, p.tiles_per_split, C, ct, K, w.pR, w.pD, w.pK, w.xn2,
                           nullptr, w.rlist, w.rcount, pd.corder, PruneData{}, 0.0, 0.0);
    }
    const ScreenBound b2 = screen_bound(p, src.type, ct, src.d, alpha);
    hipLaunchKernelGGL(finalize1_list_kernel, dim3(static_cast<unsigned>(cdiv(src.n, 256))), dim3(256), 0, stream,
                       p.splits, src.n, w.rlist, w.rcount, w.pR, w.pD, w.pK, w.xn2, b2, w.rcount + 1, w.rlist2,
                       out_codes, out_dist, rowD, rowK);
    // pD / pK are free once the second finalize has read them
    return launch_rescue1<2>(src, top, C, ct, K, w.rcount + 1, w.rlist2, out_codes, out_dist, rowD, rowK, w.pD, w.pK,
                             static_cast<int64_t>(p.splits) * src.n, stream);
  }
  const unsigned prep_grid = static_cast<unsigned>(cdiv(p.tiles * 16, 256));
  if (p.split) {
    hipLaunchKernelGGL(prep_codebook_split, dim3(prep_grid), dim3(256), 0, stream, C, ct, K, src.d, p.tiles,
                       reinterpret_cast<uint16_t*>(w.apack), w.cnp, w.rcount);
  } else {
    switch (p.ks) {
      case 1: hipLaunchKernelGGL(prep_codebook<1>, dim3(prep_grid), dim3(256), 0, stream, C, ct, K, src.d, p.tiles, w.apack, w.cnp, w.rcount); break;
      case 2: hipLaunchKernelGGL(prep_codebook<2>, dim3(prep_grid), dim3(256), 0, stream, C, ct, K, src.d, p.tiles, w.apack, w.cnp, w.rcount); break;
      default: hipLaunchKernelGGL(prep_codebook<4>, dim3(prep_grid), dim3(256), 0, stream, C, ct, K, src.d, p.tiles, w.apack, w.cnp, w.rcount); break;
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (p.split && top == 1 && p.splits == 1 && p.tiles <= 16) {
    // small codebook, top-1: screen, exact winner and certificate in one kernel, then the rescue
    const ScreenBound bound = screen_bound(p, src.type, ct, src.d, nullptr);
    const dim3 grid(static_cast<unsigned>(p.grid_x));
    const int ft = small1_form(src, C, ct);
#define CRVQ_SMALL1(CBV, FTV)                                                                                    \
  hipLaunchKernelGGL((screen_small1_kernel<CBV, FTV>), grid, dim3(256), 0, stream, src, w.apack, w.cnp, p.tiles, C, \
                     ct, K, bound, w.rcount, w.rlist, out_codes, out_dist, rowD, rowK)
    if (p.cb == CRVQ_CB_WIDE) {
      if (ft == 1)
        CRVQ_SMALL1(CRVQ_CB_WIDE, 1);
      else if (ft == 2)
        CRVQ_SMALL1(CRVQ_CB_WIDE, 2);
      else
        CRVQ_SMALL1(CRVQ_CB_WIDE, 0);
    } else {
      CRVQ_SMALL1(2, 0);
    }
#undef CRVQ_SMALL1
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_rescue1<2>(src, top, C, ct, K, w.rcount, w.rlist, out_codes, out_dist, rowD, rowK, nullptr, nullptr, 0,
                             stream);
  }
  if (p.split) {
    e = launch_screen_ops<SplitOps>(src, C, ct, K, p, w, stream);
  } else {
    switch (p.ks) {
      case 1: e = launch_screen_ops<F32Ops<1>>(src, C, ct, K, p, w, stream); break;
      case 2: e = launch_screen_ops<F32Ops<2>>(src, C, ct, K, p, w, stream); break;
      default: e = launch_screen_ops<F32Ops<4>>(src, C, ct, K, p, w, stream); break;
    }
  }
  if (e != hipSuccess) return e;
  const ScreenBound bound = screen_bound(p, src.type, ct, src.d, nullptr);
  switch (p.ks) {
    case 1: return launch_finalize_ks<1>(src, C, ct, K, top, p, w, bound, out_codes, out_dist, rowD, rowK, stream);
    case 2: return launch_finalize_ks<2>(src, C, ct, K, top, p, w, bound, out_codes, out_dist, rowD, rowK, stream);
    default: return launch_finalize_ks<4>(src, C, ct, K, top, p, w, bound, out_codes, out_dist, rowD, rowK, stream);
  }
}

hipError_t launch_beam_merge(int64_t n, int n_par, int beam, int step, int n_books, const double* rowD,
                             const int* rowK, const RowSrc& src0, const double* res_in, double* res_out,
                             const int* tup_in, int* tup_out, double* err_out, const void* book, int book_type,
                             int64_t K, int d, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t nn = static_cast<int64_t>(n_par) * K;
  const int n_next = static_cast<int>(nn < beam ? nn : beam);
  if (n_par * beam > 1 && n_par <= 8 && beam <= 8) {  // a real merge: eight lanes per vector
    hipLaunchKernelGGL(beam_merge_lanes, dim3(static_cast<unsigned>(cdiv(n, 32))), dim3(256), 0, stream, n, n_par,
                       n_next, beam, step, n_books, rowD, rowK, src0, res_in, res_out, tup_in, tup_out, err_out, book,
                       book_type, K, d);
  } else if (n_par * beam > 1) {  // wider beams: one wave per vector
    hipLaunchKernelGGL(beam_merge_wave, dim3(static_cast<unsigned>(cdiv(n, 4))), dim3(256), 0, stream, n, n_par,
                       n_next, beam, step, n_books, rowD, rowK, src0, res_in, res_out, tup_in, tup_out, err_out, book,
                       book_type, K, d);
  } else {
    hipLaunchKernelGGL(beam_merge_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0, stream, n, n_par,
                       n_next, beam, step, n_books, rowD, rowK, src0, res_in, res_out, tup_in, tup_out, err_out, book,
                       book_type, K, d);
  }
  return hipGetLastError();
}

hipError_t launch_beam_emit(int64_t n, int64_t vpr, int n_par, int n_books, const int* tup, const double* err,
                            const CodePtrs& outs, float* err_out, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(beam_emit_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0, stream, n, vpr, n_par,
                     n_books, tup, err, outs, err_out);
  return hipGetLastError();
}

}  // namespace crvq
