// Lloyd update of a K-means codebook (Sec. 3.1 Eq. 2 of the paper; Alg. 1 KMeansCodebook):
// every centroid becomes the mean of the vectors encoded to it.
//
// Deterministic: every centroid is a fixed-order fp64 sum of its members (no floating-point
// atomics), divided by their count and rounded once to the codebook's type; a codeword without
// members is left untouched; codes outside [0, K) belong to no cluster.  Only the radix histogram
// counts with integer LDS atomics.
// * K <= 256 (small_k_partial): blocks walk contiguous vector ranges; each round of 1024 codes is
//   bucket-sorted in LDS and thread k adds the members of code k.
// * K > 256 (bucket_partial8 / bucket_partial): one stable radix pass (per-tile ballot counting,
//   device-wide scan, stable scatter -- no atomics) groups the vectors by the high byte of their
//   code; each bucket is then reduced like a small codebook on the low byte, its member vectors
//   gathered a round at a time into LDS.  Buckets are cut into chunks taken in chunk-major order,
//   so the blocks in flight read about the same index range of every bucket.
#include "crvq_internal.h"

namespace crvq {
namespace {

constexpr int kTile = 4096;        // keys per radix tile: 4 waves x 16 batches x 64 lanes
constexpr int kBatches = 16;
constexpr int kScanBlock = 4096;   // elements per scan block: 256 threads x 16

__device__ __forceinline__ float bf16_to_f(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

__device__ __forceinline__ int64_t row_offset(const RowSrc& s, int64_t i) {
  if (s.ld == s.vpr * s.d) return i * s.d;  // rows packed back to back
  const uint32_t r = static_cast<uint32_t>(i) / static_cast<uint32_t>(s.vpr);
  const uint32_t g = static_cast<uint32_t>(i) - r * static_cast<uint32_t>(s.vpr);
  return static_cast<int64_t>(r) * s.ld + static_cast<int64_t>(g) * s.d;
}

__device__ __forceinline__ double row_elem(const RowSrc& s, int64_t off, int t) {
  if (s.type == ET_F32) return static_cast<double>(static_cast<const float*>(s.base)[off + t]);
  if (s.type == ET_F64) return static_cast<const double*>(s.base)[off + t];
  return static_cast<double>(bf16_to_f(static_cast<const uint16_t*>(s.base)[off + t]));
}

// Round an fp64 value to bfloat16, nearest-even, working on the fp64 bit pattern (no detour
// through fp32, which could round twice).
__device__ __forceinline__ uint16_t bf16_from_double(double x) {
  const double ax = fabs(x);
  if (!(ax >= 0x1p-126)) {  // zero or below the smallest normal: fixed quantum 2^-133
    const double r = rint(x * 0x1p133) * 0x1p-133;
    return static_cast<uint16_t>(__float_as_uint(static_cast<float>(r)) >> 16);
  }
  uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
  const uint64_t lsb = (u >> 45) & 1;  // 52 - 7 fraction bits are dropped
  u += (1ull << 44) - 1 + lsb;
  u &= ~((1ull << 45) - 1);
  const float f = static_cast<float>(__longlong_as_double(static_cast<long long>(u)));  // exact or +-inf
  return static_cast<uint16_t>(__float_as_uint(f) >> 16);
}

// Lanes of this wave whose (valid, digit) equals ours.
__device__ __forceinline__ uint64_t peer_mask(bool valid, int digit) {
  uint64_t peers = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (digit >> b) & 1;
    const uint64_t m = __ballot(bit);
    peers &= bit ? m : ~m;
  }
  return valid ? peers : 0ull;
}

__device__ __forceinline__ int read_count(const int* n_dev, int64_t n_host) {
  return n_dev ? *n_dev : static_cast<int>(n_host);
}

// ---- device-wide exclusive scan of int32 ---------------------------------------------------------
__device__ __forceinline__ int block_exclusive_scan(int v, int* sh, int& total) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    int t = (tid >= off) ? sh[tid - off] : 0;
    __syncthreads();
    sh[tid] += t;
    __syncthreads();
  }
  total = sh[255];
  const int excl = sh[tid] - v;
  __syncthreads();
  return excl;
}

// Per-tile digit counts, hist[digit * n_tiles + tile].
__global__ __launch_bounds__(256) void radix_hist(const int* __restrict__ keys, const int* __restrict__ n_dev,
                                                  int64_t n_host, int64_t K, int pass, int shift, int64_t n_tiles,
                                                  int* __restrict__ hist) {
  __shared__ int wh[4][256];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int b = tid; b < 1024; b += 256) (&wh[0][0])[b] = 0;
  __syncthreads();
  const int n = read_count(n_dev, n_host);
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kTile + w * (kBatches * 64);
  int key[kBatches];
#pragma unroll
  for (int bt = 0; bt < kBatches; ++bt) {  // every load issued before the first is counted
    const int64_t idx = base + bt * 64 + lane;
    key[bt] = (idx < n) ? ld_stream_i32(keys + idx) : -1;
  }
  // counting only (no ranks): integer LDS atomics, whose totals do not depend on their order
#pragma unroll
  for (int bt = 0; bt < kBatches; ++bt) {
    const int64_t idx = base + bt * 64 + lane;
    const bool valid = (idx < n) && (pass != 0 || (key[bt] >= 0 && key[bt] < K));
    if (valid) atomicAdd(&wh[w][(key[bt] >> shift) & 255], 1);
  }
  __syncthreads();
  hist[static_cast<int64_t>(tid) * n_tiles + blockIdx.x] = wh[0][tid] + wh[1][tid] + wh[2][tid] + wh[3][tid];
}

// Stable scatter.  The tile is first ranked into LDS by digit -- rank = (earlier waves of the tile)
// + (earlier batches of this wave) + (lower lanes) -- and then copied out in LDS order, so every
// digit's run of the tile is written to consecutive global positions.
__global__ __launch_bounds__(256) void radix_scatter(const int* __restrict__ keys_in, const int* __restrict__ vals_in,
                                                     const int* __restrict__ n_dev, int64_t n_host, int64_t K, int pass,
                                                     int shift, int64_t n_tiles, const int* __restrict__ offsets,
                                                     int* __restrict__ keys_out, int* __restrict__ vals_out) {
  __shared__ int wh[4][256];
  __shared__ int dstart[257];
  __shared__ int gstart[256];
  __shared__ int sh[256];
  __shared__ int lkey[kTile];
  __shared__ int lval[kTile];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int b = tid; b < 1024; b += 256) (&wh[0][0])[b] = 0;
  __syncthreads();
  const int n = read_count(n_dev, n_host);
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kTile + w * (kBatches * 64);
  int key[kBatches];
  int dig[kBatches];
  uint64_t peer[kBatches];
#pragma unroll
  for (int bt = 0; bt < kBatches; ++bt) {
    const int64_t idx = base + bt * 64 + lane;
    key[bt] = (idx < n) ? ld_stream_i32(keys_in + idx) : -1;
    const bool valid = (idx < n) && (pass != 0 || (key[bt] >= 0 && key[bt] < K));
    dig[bt] = valid ? (key[bt] >> shift) & 255 : -1;
    peer[bt] = peer_mask(valid, valid ? dig[bt] : 0);
    if (valid && (__ffsll(static_cast<long long>(peer[bt])) - 1) == lane) wh[w][dig[bt]] += __popcll(peer[bt]);
  }
  __syncthreads();
  {
    const int d = tid;
    const int tot = wh[0][d] + wh[1][d] + wh[2][d] + wh[3][d];
    int total;
    const int ds = block_exclusive_scan(tot, sh, total);
    dstart[d] = ds;
    if (d == 255) dstart[256] = total;
    gstart[d] = offsets[static_cast<int64_t>(d) * n_tiles + blockIdx.x];
    int run = ds;
    for (int ww = 0; ww < 4; ++ww) {
      const int c = wh[ww][d];
      wh[ww][d] = run;
      run += c;
    }
  }
  __syncthreads();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int bt = 0; bt < kBatches; ++bt) {
    const int64_t idx = base + bt * 64 + lane;
    if (dig[bt] >= 0) {
      const int pos = wh[w][dig[bt]] + __popcll(peer[bt] & lt);
      if (pos >= 0 && pos < kTile) {
        lkey[pos] = key[bt];
        lval[pos] = vals_in ? vals_in[idx] : static_cast<int>(idx);
      }
    }
    // every leader has read its digit's start above; now advance it
    if (dig[bt] >= 0 && (__ffsll(static_cast<long long>(peer[bt])) - 1) == lane) wh[w][dig[bt]] += __popcll(peer[bt]);
  }
  __syncthreads();
  const int T = dstart[256];
  for (int e = tid; e < T; e += 256) {
    const int k = lkey[e];
    const int dg = (k >> shift) & 255;
    const int pos = gstart[dg] + (e - dstart[dg]);
    if (pos >= 0 && pos < n) {  // always true for consistent counts; keeps every store in bounds
      keys_out[pos] = k;
      vals_out[pos] = lval[e];
    }
  }
}

__global__ __launch_bounds__(256) void scan_block_sums(const int* __restrict__ in, int64_t n, int* __restrict__ sums) {
  __shared__ int sh[256];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanBlock + threadIdx.x * 16;
  int s = 0;
  for (int j = 0; j < 16; ++j)
    if (base + j < n) s += in[base + j];
  int total;
  block_exclusive_scan(s, sh, total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(256) void scan_sums_single(int* __restrict__ sums, int64_t nb, int* __restrict__ total_out) {
  __shared__ int sh[256];
  int carry = 0;
  for (int64_t base = 0; base < nb; base += 256) {
    const int64_t i = base + threadIdx.x;
    const int v = (i < nb) ? sums[i] : 0;
    int total;
    const int ex = block_exclusive_scan(v, sh, total);
    if (i < nb) sums[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0 && total_out) *total_out = carry;
}

__global__ __launch_bounds__(256) void scan_apply(const int* __restrict__ in, int64_t n, const int* __restrict__ sums,
                                                  int* __restrict__ out) {
  __shared__ int sh[256];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanBlock + threadIdx.x * 16;
  int v[16];
  int s = 0;
  for (int j = 0; j < 16; ++j) {
    v[j] = (base + j < n) ? in[base + j] : 0;
    s += v[j];
  }
  int total;
  int run = block_exclusive_scan(s, sh, total) + sums[blockIdx.x];
  for (int j = 0; j < 16; ++j) {
    if (base + j < n) out[base + j] = run;
    run += v[j];
  }
}

__device__ __forceinline__ void store_centroid(void* C, int ct, int64_t k, int d, int t, double v) {
  if (ct == ET_F32)
    static_cast<float*>(C)[k * d + t] = static_cast<float>(v);
  else
    static_cast<uint16_t*>(C)[k * d + t] = bf16_from_double(v);
}

// ---- shared by both codebook sizes ---------------------------------------------------------------
// A "round" is up to kRound (vector, digit) entries; it is stably bucket-sorted by digit (0..255)
// in LDS with the ballot multisplit (one leader per digit and batch updates a per-wave counter, so
// no atomics): afterwards s_pos[s_start[c] .. s_start[c + 1]) lists the round's entries of digit c
// in ascending order.
constexpr int kRoundBatches = 4;
constexpr int kRound = 4 * kRoundBatches * 64;  // 1024 entries: 4 waves x 4 batches x 64 lanes

struct RoundLds {
  int s_pos[kRound];
  int s_start[257];
  int wh[4][256];
  int sh_scan[256];
};

// dig[bt] = digit of entry (wave, batch bt, lane) or -1 when absent.
__device__ __forceinline__ void round_bucket_sort(const int (&dig)[kRoundBatches], RoundLds& L,
                                                  int (*pos_out)[kRoundBatches] = nullptr) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int q = tid; q < 1024; q += 256) (&L.wh[0][0])[q] = 0;
  __syncthreads();
  uint64_t peer[kRoundBatches];
#pragma unroll
  for (int bt = 0; bt < kRoundBatches; ++bt) {
    const bool valid = dig[bt] >= 0;
    peer[bt] = peer_mask(valid, valid ? dig[bt] : 0);
    if (valid && (__ffsll(static_cast<long long>(peer[bt])) - 1) == lane) L.wh[w][dig[bt]] += __popcll(peer[bt]);
  }
  __syncthreads();
  const int tot = L.wh[0][tid] + L.wh[1][tid] + L.wh[2][tid] + L.wh[3][tid];
  L.sh_scan[tid] = tot;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int v = (tid >= off) ? L.sh_scan[tid - off] : 0;
    __syncthreads();
    L.sh_scan[tid] += v;
    __syncthreads();
  }
  const int start = L.sh_scan[tid] - tot;
  L.s_start[tid] = start;
  if (tid == 255) L.s_start[256] = L.sh_scan[255];
  int run = start;
  for (int ww = 0; ww < 4; ++ww) {
    const int c = L.wh[ww][tid];
    L.wh[ww][tid] = run;
    run += c;
  }
  __syncthreads();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int bt = 0; bt < kRoundBatches; ++bt) {
    if (dig[bt] >= 0) {
      const int pos = L.wh[w][dig[bt]] + __popcll(peer[bt] & lt);
      if (pos >= 0 && pos < kRound) L.s_pos[pos] = (w * kRoundBatches + bt) * 64 + lane;
      if (pos_out) (*pos_out)[bt] = pos;
    }
    if (dig[bt] >= 0 && (__ffsll(static_cast<long long>(peer[bt])) - 1) == lane) L.wh[w][dig[bt]] += __popcll(peer[bt]);
  }
  __syncthreads();
}

// v += vector at element offset off (d <= 16): 16-byte loads for d = 8 / 4 when aligned.
__device__ __forceinline__ void add_vector(const RowSrc& s, int64_t off, double (&v)[16]) {
  const int d = s.d;
  if (s.type == ET_F32) {
    const float* p = static_cast<const float*>(s.base) + off;
    if ((d == 8 || d == 4) && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        if (4 * q < d) {
          const float4 w = reinterpret_cast<const float4*>(p)[q];
          v[4 * q] = v[4 * q] + w.x;
          v[4 * q + 1] = v[4 * q + 1] + w.y;
          v[4 * q + 2] = v[4 * q + 2] + w.z;
          v[4 * q + 3] = v[4 * q + 3] + w.w;
        }
      }
      return;
    }
  } else if (s.type == ET_BF16 && d == 8 &&
             (reinterpret_cast<uintptr_t>(static_cast<const uint16_t*>(s.base) + off) & 15) == 0) {
    const uint4 w = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(s.base) + off);
    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[2 * q] = v[2 * q] + __uint_as_float(u[q] << 16);
      v[2 * q + 1] = v[2 * q + 1] + __uint_as_float(u[q] & 0xffff0000u);
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < 16; ++t)
    if (t < d) v[t] = v[t] + row_elem(s, off, t);
}

// ---- small codebooks (K <= 256): one thread per code, no global sort ------------------------------
// Each block walks a contiguous range of vectors in rounds of kRound.  A round's vectors are staged
// in LDS with coalesced loads when the set is contiguous and d <= 8; its codes are bucket-sorted and
// thread k adds the members of code k in ascending order to fp64 accumulators.  The per-block
// partials (layout [k][t][block]) are folded in block order by one wave per centroid element.
__global__ __launch_bounds__(256) void small_k_partial(RowSrc src, const int32_t* __restrict__ codes, int64_t K,
                                                       int64_t per_block, int staged, int64_t nblocks,
                                                       double* __restrict__ part, int* __restrict__ pcount) {
  __shared__ RoundLds L;
  __shared__ float s_vec[kRound * 8];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int d = src.d;
  const int64_t n = src.n;
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per_block;
  const int64_t b1 = (b0 + per_block < n) ? b0 + per_block : n;
  double acc[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) acc[t] = 0.0;
  int cnt = 0;
  for (int64_t base = b0; base < b1; base += kRound) {
    const int rn = static_cast<int>((b1 - base) < kRound ? (b1 - base) : kRound);
    if (staged) {  // vectors base .. base + rn are contiguous: one vector per thread and step
      for (int v = tid; v < rn; v += 256) {
        double tmp[16];
#pragma unroll
        for (int t = 0; t < 16; ++t) tmp[t] = 0.0;
        add_vector(src, (base + v) * d, tmp);
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (t < d) s_vec[v * d + t] = static_cast<float>(tmp[t]);
      }
    }
    int dig[kRoundBatches];
#pragma unroll
    for (int bt = 0; bt < kRoundBatches; ++bt) {
      const int e = (w * kRoundBatches + bt) * 64 + lane;
      const int c = (e < rn) ? codes[base + e] : -1;
      dig[bt] = (c >= 0 && c < K) ? c : -1;
    }
    round_bucket_sort(dig, L);  // ends with a barrier, so s_vec is complete too
    if (tid < K) {
      const int e = L.s_start[tid + 1];
      for (int j = L.s_start[tid]; j < e; ++j) {
        const int v = L.s_pos[j];
        if (staged) {
#pragma unroll
          for (int t = 0; t < 8; ++t)
            if (t < d) acc[t] = acc[t] + static_cast<double>(s_vec[v * d + t]);
        } else {
          add_vector(src, row_offset(src, base + v), acc);
        }
      }
      cnt += e - L.s_start[tid];
    }
    __syncthreads();
  }
  if (tid < K) {
#pragma unroll
    for (int t = 0; t < 16; ++t)
      if (t < d) part[(static_cast<int64_t>(tid) * d + t) * nblocks + blockIdx.x] = acc[t];
    pcount[static_cast<int64_t>(tid) * nblocks + blockIdx.x] = cnt;
  }
}

// ---- small codebooks, d <= 8: per-wave tables, no sort ------------------------------------------
// Every wave owns a private fp64 table of K x 8 sums in LDS and the batches of 64 vectors
// j = wave, wave + W, wave + 2W, ... (W waves in the grid), so the waves in flight read one moving
// window of memory.  It reads one vector per lane, kSkDepth batches in flight; within a batch the
// lanes that share a code find each other with eight ballots, and the lowest of them adds its peers'
// vectors (staged in LDS) to the table entry of that code in ascending order.  So every table entry
// is a fixed-order sequential sum of its code's members over the wave's batches.  At the end the
// block folds its wave tables in wave order into one partial per block (layout [k][t][block]);
// small_k_final folds those in block order.
constexpr int kSkWaves = 8;
constexpr int kSkDepth = 4;

// LDS layout of a wave's table and stage.  Sum t of code c sits at c * 8 + (t ^ ((c >> 1) & 7)): with
// the plain c * 8 + t, the 64 lanes of a batch (one code each) read dimension t from only two 8-byte
// bank pairs of the 32 banks (codes of equal parity collide), a 32-way conflict per access; the
// swizzle spreads them over all 16 pairs.  Half h of lane l's staged vector sits at slot
// 2 l + (h ^ ((l >> 2) & 1)), so a wave's 16-byte stores and loads cover every bank.
__device__ __forceinline__ int sk_slot(int c, int t) { return c * 8 + (t ^ ((c >> 1) & 7)); }
__device__ __forceinline__ int sk_stage(int l, int h) { return 2 * l + (h ^ ((l >> 2) & 1)); }

struct SkTable {
  double acc[256 * 8];
  int cnt[256];
  float4 stage[64][2];
};

// Vector i as 8 floats (zero past d).  KIND 0: fp32 d = 8 with 16-byte aligned vectors (two
// nontemporal 16-byte loads), KIND 1: bf16 d = 8 aligned (one), KIND 2: element loads (any d <= 8).
// KIND 0 / 1 are straight-line code: a lane outside the range reads vector 0 (its code is set to
// -1, so the values are never used), which keeps every prefetched batch in flight.
template <int KIND>
__device__ __forceinline__ void sk_load(const RowSrc& s, int64_t i, bool ok, float4& a, float4& b) {
  const int64_t off = row_offset(s, ok ? i : 0);
  if constexpr (KIND == 0) {
    const float* p = static_cast<const float*>(s.base) + off;
    const uint4 x = ld_stream(p), y = ld_stream(p + 4);
    a = make_float4(__uint_as_float(x.x), __uint_as_float(x.y), __uint_as_float(x.z), __uint_as_float(x.w));
    b = make_float4(__uint_as_float(y.x), __uint_as_float(y.y), __uint_as_float(y.z), __uint_as_float(y.w));
  } else if constexpr (KIND == 1) {
    const uint4 q = ld_stream(static_cast<const uint16_t*>(s.base) + off);
    a = make_float4(__uint_as_float(q.x << 16), __uint_as_float(q.x & 0xffff0000u), __uint_as_float(q.y << 16),
                    __uint_as_float(q.y & 0xffff0000u));
    b = make_float4(__uint_as_float(q.z << 16), __uint_as_float(q.z & 0xffff0000u), __uint_as_float(q.w << 16),
                    __uint_as_float(q.w & 0xffff0000u));
  } else {
    float e[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) e[t] = (ok && t < s.d) ? static_cast<float>(row_elem(s, off, t)) : 0.0f;
    a = make_float4(e[0], e[1], e[2], e[3]);
    b = make_float4(e[4], e[5], e[6], e[7]);
  }
}

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int KIND>
__global__ __launch_bounds__(64 * kSkWaves) void small_k_wave_partial(RowSrc src, const int32_t* __restrict__ codes,
                                                                       int64_t K, int64_t per_wave, int64_t nblocks,
                                                                       double* __restrict__ part,
                                                                       int* __restrict__ pcount) {
  __shared__ SkTable tab[kSkWaves];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  SkTable& T = tab[w];
  const int d = src.d;
  for (int e = lane; e < 256 * 8; e += 64) T.acc[e] = 0.0;
  for (int e = lane; e < 256; e += 64) T.cnt[e] = 0;
  const int64_t n = src.n;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kSkWaves * 64;  // elements between a wave's batches
  const int64_t w0 = (static_cast<int64_t>(blockIdx.x) * kSkWaves + w) * 64;
  const int64_t w1 = n;
  (void)per_wave;
  // kSkDepth batches in flight: slot s holds batch base + 64 s and is refilled right after use
  // with the batch kSkDepth further on (the loop is unrolled over the slots, so no register holding
  // a pending load is ever copied); a lane's code is masked to -1 only when its batch is used.
  float4 va[kSkDepth], vb[kSkDepth];
  int cq[kSkDepth];
#pragma unroll
  for (int s = 0; s < kSkDepth; ++s) {
    const int64_t i = w0 + stride * s + lane;
    const bool ok = i < w1;
    sk_load<KIND>(src, i, ok, va[s], vb[s]);
    cq[s] = ld_stream_i32(codes + (ok ? i : 0));
  }
  for (int64_t base = w0; base < w1; base += stride * kSkDepth) {
#pragma unroll
    for (int s = 0; s < kSkDepth; ++s) {
      const int64_t bb = base + stride * s;
      if (bb < w1) {  // uniform
        const int c = (bb + lane < w1) ? cq[s] : -1;
        const bool valid = c >= 0 && c < K;
        (&T.stage[0][0])[sk_stage(lane, 0)] = va[s];
        (&T.stage[0][0])[sk_stage(lane, 1)] = vb[s];
        wave_lds_sync();  // staged vectors and the previous batch's table updates are visible
        const uint64_t peers = peer_mask(valid, valid ? c : 0);
        if (valid && (__ffsll(static_cast<long long>(peers)) - 1) == lane) {
          double acc[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) acc[t] = T.acc[sk_slot(c, t)];
          uint64_t m = peers;
          while (m) {
            const int sl = __ffsll(static_cast<long long>(m)) - 1;
            m &= m - 1;
            const float4 x0 = (&T.stage[0][0])[sk_stage(sl, 0)], x1 = (&T.stage[0][0])[sk_stage(sl, 1)];
            const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
            for (int t = 0; t < 8; ++t) acc[t] = acc[t] + static_cast<double>(x[t]);
          }
#pragma unroll
          for (int t = 0; t < 8; ++t) T.acc[sk_slot(c, t)] = acc[t];
          T.cnt[c] += __popcll(peers);
        }
        wave_lds_sync();  // the stage is rewritten by the next batch
      }
      const int64_t i = bb + stride * kSkDepth + lane;
      const bool ok = i < w1;
      sk_load<KIND>(src, i, ok, va[s], vb[s]);
      cq[s] = ld_stream_i32(codes + (ok ? i : 0));
    }
  }
  __syncthreads();
  for (int64_t e = tid; e < K * d; e += 64 * kSkWaves) {
    const int64_t k = e / d;
    const int t = static_cast<int>(e - k * d);
    double acc = 0.0;
#pragma unroll
    for (int ww = 0; ww < kSkWaves; ++ww) acc = acc + tab[ww].acc[sk_slot(static_cast<int>(k), t)];
    part[e * nblocks + blockIdx.x] = acc;
    if (t == 0) {
      int cnt = 0;
#pragma unroll
      for (int ww = 0; ww < kSkWaves; ++ww) cnt += tab[ww].cnt[k];
      pcount[k * nblocks + blockIdx.x] = cnt;
    }
  }
}

// One wave per centroid element: lanes fold blocks lane, lane + 64, ... in order, then a fixed
// xor butterfly (the same in every lane).
__global__ __launch_bounds__(256) void small_k_final(const double* __restrict__ part, const int* __restrict__ pcount,
                                                     int64_t nblocks, int64_t K, int d, void* C, int ct,
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
    if (counts && t == 0) counts[k] = cnt;
    if (cnt > 0) store_centroid(C, ct, k, d, t, acc / static_cast<double>(cnt));
  }
}

struct SmallPlan {
  int64_t blocks;
  int64_t per_block;
};

// The per-wave scheme: one block of kSkWaves waves per CU (LDS holds one block), at most one wave
// per batch of 64 vectors.
SmallPlan wave_plan(int64_t n) {
  SmallPlan p;
  const int64_t batches = cdiv(n > 0 ? n : 1, 64);
  const int64_t waves = batches < 256 * kSkWaves ? batches : 256 * kSkWaves;
  p.blocks = cdiv(waves, kSkWaves);
  p.per_block = 64;
  return p;
}

SmallPlan small_plan(int64_t n) {
  SmallPlan p;
  const int64_t rounds = cdiv(n > 0 ? n : 1, kRound);
  p.blocks = rounds < 2048 ? rounds : 2048;
  p.per_block = cdiv(rounds, p.blocks) * kRound;
  p.blocks = cdiv(n > 0 ? n : 1, p.per_block);
  return p;
}

// ---- large codebooks (256 < K <= 65536) ----------------------------------------------------------
// One stable radix pass groups the vectors by the high byte of their code (256 buckets of 256 codes).
// Every bucket is then cut into chunks of kChunk vectors; a block takes one chunk and runs the
// small-codebook scheme on the low byte, gathering each member vector with 16-byte loads.  The
// chunk partials of each code are folded in chunk order.
#ifndef CRVQ_KM_CHUNK
#define CRVQ_KM_CHUNK 4096
#endif
constexpr int kChunk = CRVQ_KM_CHUNK;

// bounds of the 256 high-byte buckets and of their chunk ranges (one block)
// Chunks are also enumerated level by level (chunk j of every bucket that has one, buckets in
// ascending order, before any chunk j + 1): lstart[j] = number of chunks below level j, for
// j = 0 .. max_level, where level j holds the buckets with more than j chunks.  Blocks take the
// chunks in that order, so the blocks in flight read vectors from about the same index range of
// every bucket at once.
__global__ __launch_bounds__(256) void bucket_bounds(const int* __restrict__ offs, int64_t n_tiles,
                                                     const int* __restrict__ n_valid, int* __restrict__ bstart,
                                                     int* __restrict__ cstart, int* __restrict__ lstart) {
  __shared__ int sh[256];
  __shared__ int nch[256];
  __shared__ int maxc;
  const int b = threadIdx.x;
  const int s = offs[static_cast<int64_t>(b) * n_tiles];
  const int e = (b < 255) ? offs[static_cast<int64_t>(b + 1) * n_tiles] : *n_valid;
  const int chunks = (e - s + kChunk - 1) / kChunk;
  int total;
  const int ex = block_exclusive_scan(chunks, sh, total);
  bstart[b] = s;
  cstart[b] = ex;
  if (b == 255) {
    bstart[256] = e;
    cstart[256] = total;
  }
  nch[b] = chunks;
  if (b == 0) maxc = 0;
  __syncthreads();
  if (b == 0) {
    int m = 0;
    for (int q = 0; q < 256; ++q) m = nch[q] > m ? nch[q] : m;
    maxc = m;
  }
  __syncthreads();
  const int levels = maxc;
  int carry = 0;
  for (int j0 = 0; j0 < levels; j0 += 256) {
    const int j = j0 + b;
    int cnt = 0;
    if (j < levels)
      for (int q = 0; q < 256; ++q) cnt += (nch[q] > j) ? 1 : 0;
    int tot;
    const int lex = block_exclusive_scan(cnt, sh, tot);
    if (j < levels) lstart[j] = carry + lex;
    carry += tot;
  }
  if (b == 0) lstart[levels] = carry;  // == total
  if (b == 0) cstart[257] = levels;
}

__global__ __launch_bounds__(256) void bucket_partial(RowSrc src, const int* __restrict__ keys,
                                                      const int* __restrict__ vals, const int* __restrict__ bstart,
                                                      const int* __restrict__ cstart, double* __restrict__ part,
                                                      int* __restrict__ pcount) {
  __shared__ RoundLds L;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int blk = blockIdx.x;
  if (blk >= cstart[256]) return;  // uniform: more blocks are launched than there can be chunks
  int lo = 0, hi = 256;            // bucket b with cstart[b] <= blk < cstart[b + 1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cstart[mid] <= blk)
      lo = mid;
    else
      hi = mid;
  }
  const int b = lo;
  const int64_t b0 = bstart[b] + static_cast<int64_t>(blk - cstart[b]) * kChunk;
  const int64_t b1 = (b0 + kChunk < bstart[b + 1]) ? b0 + kChunk : bstart[b + 1];
  const int d = src.d;
  double acc[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) acc[t] = 0.0;
  int cnt = 0;
  for (int64_t base = b0; base < b1; base += kRound) {
    int dig[kRoundBatches];
#pragma unroll
    for (int bt = 0; bt < kRoundBatches; ++bt) {
      const int64_t idx = base + (w * kRoundBatches + bt) * 64 + lane;
      dig[bt] = (idx < b1) ? (keys[idx] & 255) : -1;
    }
    round_bucket_sort(dig, L);
    const int e = L.s_start[tid + 1];
    int j = L.s_start[tid];
    for (; j + 1 < e; j += 2) {  // two members' loads in flight, added in ascending order
      double v0[16], v1[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        v0[t] = 0.0;
        v1[t] = 0.0;
      }
      add_vector(src, row_offset(src, vals[base + L.s_pos[j]]), v0);
      add_vector(src, row_offset(src, vals[base + L.s_pos[j + 1]]), v1);
#pragma unroll
      for (int t = 0; t < 16; ++t)
        if (t < d) acc[t] = (acc[t] + v0[t]) + v1[t];
    }
    if (j < e) add_vector(src, row_offset(src, vals[base + L.s_pos[j]]), acc);
    cnt += e - L.s_start[tid];
    __syncthreads();
  }
  double* pp = part + (static_cast<int64_t>(blk) * 256 + tid) * d;
#pragma unroll
  for (int t = 0; t < 16; ++t)
    if (t < d) pp[t] = acc[t];
  pcount[static_cast<int64_t>(blk) * 256 + tid] = cnt;
}

// d <= 8: a round's member vectors are gathered all at once (kRoundBatches per thread, every load
// issued before any is used) into LDS at their sorted position; thread k then adds the members of
// code k from LDS in ascending order -- the same fp64 additions in the same order as above.
__global__ __launch_bounds__(256) void bucket_partial8(RowSrc src, const int* __restrict__ keys,
                                                       const int* __restrict__ vals, const int* __restrict__ bstart,
                                                       const int* __restrict__ cstart, const int* __restrict__ lstart,
                                                       double* __restrict__ part, int* __restrict__ pcount) {
  __shared__ RoundLds L;
  __shared__ float4 stage[kRound][2];
  __shared__ int s_bucket;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wi = blockIdx.x;
  if (wi >= cstart[256]) return;  // uniform: more blocks are launched than there can be chunks
  // level j of work item wi, then the (wi - lstart[j])-th bucket with more than j chunks
  const int levels = cstart[257];
  int lo = 0, hi = levels;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (lstart[mid] <= wi)
      lo = mid;
    else
      hi = mid;
  }
  const int j = lo;
  const int rank = wi - lstart[j];
  {
    const int has = (cstart[tid + 1] - cstart[tid]) > j ? 1 : 0;
    int tot;
    const int before = block_exclusive_scan(has, L.sh_scan, tot);
    if (has && before == rank) s_bucket = tid;
    __syncthreads();
  }
  const int b = s_bucket;
  const int blk = cstart[b] + j;  // partials stay in bucket-major order
  const int64_t b0 = bstart[b] + static_cast<int64_t>(j) * kChunk;
  const int64_t b1 = (b0 + kChunk < bstart[b + 1]) ? b0 + kChunk : bstart[b + 1];
  const int d = src.d;
  const bool packed = src.ld == src.vpr * d;
  double acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = 0.0;
  int cnt = 0;
  for (int64_t base = b0; base < b1; base += kRound) {
    int dig[kRoundBatches], vid[kRoundBatches], pos[kRoundBatches];
#pragma unroll
    for (int bt = 0; bt < kRoundBatches; ++bt) {
      const int64_t idx = base + (w * kRoundBatches + bt) * 64 + lane;
      const bool live = idx < b1;
      dig[bt] = live ? (ld_stream_i32(keys + idx) & 255) : -1;
      vid[bt] = live ? ld_stream_i32(vals + idx) : -1;
    }
    round_bucket_sort(dig, L, &pos);
    float4 v[kRoundBatches][2];
#pragma unroll
    for (int bt = 0; bt < kRoundBatches; ++bt) {
      v[bt][0] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      v[bt][1] = v[bt][0];
      if (vid[bt] >= 0) {
        const int64_t off = packed ? static_cast<int64_t>(vid[bt]) * d : row_offset(src, vid[bt]);
        if (src.type == ET_F32 && d == 8 && (reinterpret_cast<uintptr_t>(static_cast<const float*>(src.base) + off) & 15) == 0) {
          const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(src.base) + off);
          v[bt][0] = p[0];
          v[bt][1] = p[1];
        } else if (src.type == ET_BF16 && d == 8 &&
                   (reinterpret_cast<uintptr_t>(static_cast<const uint16_t*>(src.base) + off) & 15) == 0) {
          const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(src.base) + off);
          v[bt][0] = make_float4(__uint_as_float(q.x << 16), __uint_as_float(q.x & 0xffff0000u),
                                 __uint_as_float(q.y << 16), __uint_as_float(q.y & 0xffff0000u));
          v[bt][1] = make_float4(__uint_as_float(q.z << 16), __uint_as_float(q.z & 0xffff0000u),
                                 __uint_as_float(q.w << 16), __uint_as_float(q.w & 0xffff0000u));
        } else {
          float e[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) e[t] = (t < d) ? static_cast<float>(row_elem(src, off, t)) : 0.0f;
          v[bt][0] = make_float4(e[0], e[1], e[2], e[3]);
          v[bt][1] = make_float4(e[4], e[5], e[6], e[7]);
        }
      }
    }
#pragma unroll
    for (int bt = 0; bt < kRoundBatches; ++bt) {
      if (vid[bt] >= 0 && pos[bt] >= 0 && pos[bt] < kRound) {
        stage[pos[bt]][0] = v[bt][0];
        stage[pos[bt]][1] = v[bt][1];
      }
    }
    __syncthreads();
    const int e1 = L.s_start[tid + 1];
    for (int j = L.s_start[tid]; j < e1; ++j) {
      const float4 a = stage[j][0], c = stage[j][1];
      const float x[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (t < d) acc[t] = acc[t] + static_cast<double>(x[t]);
    }
    cnt += e1 - L.s_start[tid];
    __syncthreads();
  }
  double* pp = part + (static_cast<int64_t>(blk) * 256 + tid) * d;
#pragma unroll
  for (int t = 0; t < 8; ++t)
    if (t < d) pp[t] = acc[t];
  pcount[static_cast<int64_t>(blk) * 256 + tid] = cnt;
}

__global__ __launch_bounds__(256) void bucket_final(const double* __restrict__ part, const int* __restrict__ pcount,
                                                    const int* __restrict__ cstart, int64_t K, int d, void* C, int ct,
                                                    int32_t* __restrict__ counts) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= K * d) return;
  const int64_t k = e / d;
  const int t = static_cast<int>(e - k * d);
  const int b = static_cast<int>(k >> 8), low = static_cast<int>(k & 255);
  double acc = 0.0;
  int cnt = 0;
  for (int blk = cstart[b]; blk < cstart[b + 1]; ++blk) {
    acc = acc + part[(static_cast<int64_t>(blk) * 256 + low) * d + t];
    cnt += pcount[static_cast<int64_t>(blk) * 256 + low];
  }
  if (counts && t == 0) counts[k] = cnt;
  if (cnt > 0) store_centroid(C, ct, k, d, t, acc / static_cast<double>(cnt));
}

// Per-code sums and counts instead of means (the gradient sums of the codebook fine-tuning).
__global__ __launch_bounds__(256) void bucket_final_sums(const double* __restrict__ part, const int* __restrict__ pcount,
                                                         const int* __restrict__ cstart, int64_t K, int d,
                                                         double* __restrict__ sums, int32_t* __restrict__ counts) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= K * d) return;
  const int64_t k = e / d;
  const int t = static_cast<int>(e - k * d);
  const int b = static_cast<int>(k >> 8), low = static_cast<int>(k & 255);
  double acc = 0.0;
  int cnt = 0;
  for (int blk = cstart[b]; blk < cstart[b + 1]; ++blk) {
    acc = acc + part[(static_cast<int64_t>(blk) * 256 + low) * d + t];
    cnt += pcount[static_cast<int64_t>(blk) * 256 + low];
  }
  sums[e] = acc;
  if (counts && t == 0) counts[k] = cnt;
}

struct KmWs {
  int* keys;
  int* vals;
  int* hist;
  int* offs;
  int* sums;
  int* n_valid;
  int* bstart;
  int* cstart;
  int* lstart;
  double* part;
  int* pcount;
  int64_t max_chunks;
};

KmWs carve(WsCursor& ws, int64_t n, int64_t K) {
  (void)K;
  KmWs w;
  const int64_t n_tiles = cdiv(n > 0 ? n : 1, kTile);
  const int64_t hn = 256 * n_tiles;
  w.keys = ws.take<int>(static_cast<size_t>(n));
  w.vals = ws.take<int>(static_cast<size_t>(n));
  w.hist = ws.take<int>(static_cast<size_t>(hn));
  w.offs = ws.take<int>(static_cast<size_t>(hn));
  w.sums = ws.take<int>(static_cast<size_t>(cdiv(hn, kScanBlock)));
  w.n_valid = ws.take<int>(1);
  w.bstart = ws.take<int>(257);
  w.cstart = ws.take<int>(258);  // [256] = chunks, [257] = levels
  w.max_chunks = cdiv(n, kChunk) + 256;  // every bucket adds at most one partial chunk
  w.lstart = ws.take<int>(static_cast<size_t>(w.max_chunks + 1));
  w.part = ws.take<double>(static_cast<size_t>(w.max_chunks) * 256 * 16);
  w.pcount = ws.take<int>(static_cast<size_t>(w.max_chunks) * 256);
  return w;
}

hipError_t exclusive_scan(const int* in, int64_t n, int* sums, int* out, int* total, hipStream_t stream) {
  const int64_t nb = cdiv(n, kScanBlock);
  hipLaunchKernelGGL(scan_block_sums, dim3(static_cast<unsigned>(nb)), dim3(256), 0, stream, in, n, sums);
  hipLaunchKernelGGL(scan_sums_single, dim3(1), dim3(256), 0, stream, sums, nb, total);
  hipLaunchKernelGGL(scan_apply, dim3(static_cast<unsigned>(nb)), dim3(256), 0, stream, in, n, sums, out);
  return hipGetLastError();
}

}  // namespace

size_t kmeans_ws_bytes(int64_t n, int64_t K) {
  WsCursor c(nullptr);
  if (K <= 256) {
    SmallPlan p = small_plan(n), q = wave_plan(n);
    const int64_t blocks = p.blocks > q.blocks ? p.blocks : q.blocks;
    c.take<double>(static_cast<size_t>(blocks * K * 16));
    c.take<int>(static_cast<size_t>(blocks * K));
    return c.used;
  }
  carve(c, n, K);
  return c.used;
}

size_t code_sums_large_ws_bytes(int64_t n, int64_t K) {
  WsCursor c(nullptr);
  carve(c, n, K);
  return c.used;
}

// Per-code sums of the vectors of src (any element type, d <= 16) for 256 < K <= 65536: the radix
// grouping of the large-codebook K-means update, with sums and counts as the result.  Every code's
// members are added in ascending vector order within a chunk of its bucket, the chunks in order.
hipError_t launch_code_sums_large(const RowSrc& src, const int32_t* codes, int64_t K, double* sums, int32_t* counts,
                                  void* ws, hipStream_t stream) {
  const int64_t n = src.n;
  WsCursor cur(ws);
  KmWs w = carve(cur, n, K);
  const int64_t n_tiles = cdiv(n > 0 ? n : 1, kTile);
  hipError_t e;
  hipLaunchKernelGGL(radix_hist, dim3(static_cast<unsigned>(n_tiles)), dim3(256), 0, stream, codes, nullptr, n, K, 0, 8,
                     n_tiles, w.hist);
  if ((e = exclusive_scan(w.hist, 256 * n_tiles, w.sums, w.offs, w.n_valid, stream)) != hipSuccess) return e;
  hipLaunchKernelGGL(radix_scatter, dim3(static_cast<unsigned>(n_tiles)), dim3(256), 0, stream, codes, nullptr, nullptr,
                     n, K, 0, 8, n_tiles, w.offs, w.keys, w.vals);
  hipLaunchKernelGGL(bucket_bounds, dim3(1), dim3(256), 0, stream, w.offs, n_tiles, w.n_valid, w.bstart, w.cstart,
                     w.lstart);
  hipLaunchKernelGGL(bucket_partial, dim3(static_cast<unsigned>(w.max_chunks)), dim3(256), 0, stream, src, w.keys,
                     w.vals, w.bstart, w.cstart, w.part, w.pcount);
  hipLaunchKernelGGL(bucket_final_sums, dim3(static_cast<unsigned>(cdiv(K * src.d, 256))), dim3(256), 0, stream,
                     w.part, w.pcount, w.cstart, K, src.d, sums, counts);
  return hipGetLastError();
}

hipError_t launch_kmeans_update(const RowSrc& src, const int32_t* codes, int64_t K, void* C, int c_type,
                                int32_t* counts, void* ws, hipStream_t stream) {
  const int64_t n = src.n;
  WsCursor cur(ws);
  if (K <= 256) {
    SmallPlan p = small_plan(n), q = wave_plan(n);
    const int64_t blocks = p.blocks > q.blocks ? p.blocks : q.blocks;
    double* part = cur.take<double>(static_cast<size_t>(blocks * K * 16));
    int* pcount = cur.take<int>(static_cast<size_t>(blocks * K));
    if (src.d <= 8 && src.type != ET_F64 && n > 0) {
      const int es = src.type == ET_F32 ? 4 : 2;
      const bool aligned = src.d == 8 && reinterpret_cast<uintptr_t>(src.base) % 16 == 0 && (src.ld * es) % 16 == 0;
      const int kind = aligned ? (src.type == ET_F32 ? 0 : 1) : 2;
      const dim3 g3(static_cast<unsigned>(q.blocks)), b3(64 * kSkWaves);
      if (kind == 0)
        hipLaunchKernelGGL(small_k_wave_partial<0>, g3, b3, 0, stream, src, codes, K, q.per_block, q.blocks, part, pcount);
      else if (kind == 1)
        hipLaunchKernelGGL(small_k_wave_partial<1>, g3, b3, 0, stream, src, codes, K, q.per_block, q.blocks, part, pcount);
      else
        hipLaunchKernelGGL(small_k_wave_partial<2>, g3, b3, 0, stream, src, codes, K, q.per_block, q.blocks, part, pcount);
      hipLaunchKernelGGL(small_k_final, dim3(static_cast<unsigned>(cdiv(K * src.d, 4))), dim3(256), 0, stream, part,
                         pcount, q.blocks, K, src.d, C, c_type, counts);
      return hipGetLastError();
    }
    const int staged = (src.ld == src.vpr * src.d) && src.d <= 8;
    hipLaunchKernelGGL(small_k_partial, dim3(static_cast<unsigned>(p.blocks)), dim3(256), 0, stream, src, codes, K,
                       p.per_block, staged, p.blocks, part, pcount);
    hipLaunchKernelGGL(small_k_final, dim3(static_cast<unsigned>(cdiv(K * src.d, 4))), dim3(256), 0, stream, part,
                       pcount, p.blocks, K, src.d, C, c_type, counts);
    return hipGetLastError();
  }
  KmWs w = carve(cur, n, K);
  const int64_t n_tiles = cdiv(n > 0 ? n : 1, kTile);
  hipError_t e;
  hipLaunchKernelGGL(radix_hist, dim3(static_cast<unsigned>(n_tiles)), dim3(256), 0, stream, codes, nullptr, n, K, 0, 8,
                     n_tiles, w.hist);
  if ((e = exclusive_scan(w.hist, 256 * n_tiles, w.sums, w.offs, w.n_valid, stream)) != hipSuccess) return e;
  hipLaunchKernelGGL(radix_scatter, dim3(static_cast<unsigned>(n_tiles)), dim3(256), 0, stream, codes, nullptr, nullptr,
                     n, K, 0, 8, n_tiles, w.offs, w.keys, w.vals);
  hipLaunchKernelGGL(bucket_bounds, dim3(1), dim3(256), 0, stream, w.offs, n_tiles, w.n_valid, w.bstart, w.cstart,
                     w.lstart);
  if (src.d <= 8 && src.type != ET_F64)
    hipLaunchKernelGGL(bucket_partial8, dim3(static_cast<unsigned>(w.max_chunks)), dim3(256), 0, stream, src, w.keys,
                       w.vals, w.bstart, w.cstart, w.lstart, w.part, w.pcount);
  else
    hipLaunchKernelGGL(bucket_partial, dim3(static_cast<unsigned>(w.max_chunks)), dim3(256), 0, stream, src, w.keys,
                       w.vals, w.bstart, w.cstart, w.part, w.pcount);
  hipLaunchKernelGGL(bucket_final, dim3(static_cast<unsigned>(cdiv(K * src.d, 256))), dim3(256), 0, stream, w.part,
                     w.pcount, w.cstart, K, src.d, C, c_type, counts);
  return hipGetLastError();
}

}  // namespace crvq
