// Lloyd update of a K-means codebook (Sec. 3.1 Eq. 2 of the paper; Alg. 1 KMeansCodebook):
// every centroid becomes the mean of the vectors encoded to it.
//
// Atomic-free and deterministic:
// 1. the (code, vector) pairs are stably sorted by code with an LSD radix sort (8-bit digits;
//    one pass for K <= 256, two for K <= 65536).  Per 4096-key tile the digit counts and the
//    stable ranks come from wave ballots (one leader per digit and batch updates a per-wave LDS
//    counter -- no atomics), tile offsets from a device-wide exclusive scan;
// 2. the segment of every code is found by binary search in the sorted codes;
// 3. each centroid is the fixed-order fp64 reduction of its segment, divided by the count and
//    rounded once to the codebook's type; an empty segment leaves the centroid untouched.
// Codes outside [0, K) are dropped in the first pass and belong to no cluster.
// Codebooks of at most 256 codewords take a sort-free path (see small_k_partial).
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
  for (int bt = 0; bt < kBatches; ++bt) {
    const int64_t idx = base + bt * 64 + lane;
    int key = (idx < n) ? keys[idx] : -1;
    const bool valid = (idx < n) && (pass != 0 || (key >= 0 && key < K));
    const int digit = valid ? (key >> shift) & 255 : 0;
    const uint64_t peers = peer_mask(valid, digit);
    if (valid && (__ffsll(static_cast<long long>(peers)) - 1) == lane) wh[w][digit] += __popcll(peers);
  }
  __syncthreads();
  hist[static_cast<int64_t>(tid) * n_tiles + blockIdx.x] = wh[0][tid] + wh[1][tid] + wh[2][tid] + wh[3][tid];
}

// Stable scatter: rank = (earlier waves of the tile) + (earlier batches of this wave) + (lower lanes).
__global__ __launch_bounds__(256) void radix_scatter(const int* __restrict__ keys_in, const int* __restrict__ vals_in,
                                                     const int* __restrict__ n_dev, int64_t n_host, int64_t K, int pass,
                                                     int shift, int64_t n_tiles, const int* __restrict__ offsets,
                                                     int* __restrict__ keys_out, int* __restrict__ vals_out) {
  __shared__ int wh[4][256];
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
    key[bt] = (idx < n) ? keys_in[idx] : -1;
    const bool valid = (idx < n) && (pass != 0 || (key[bt] >= 0 && key[bt] < K));
    dig[bt] = valid ? (key[bt] >> shift) & 255 : -1;
    peer[bt] = peer_mask(valid, valid ? dig[bt] : 0);
    if (valid && (__ffsll(static_cast<long long>(peer[bt])) - 1) == lane) wh[w][dig[bt]] += __popcll(peer[bt]);
  }
  __syncthreads();
  // running start of every (wave, digit): tile offset + counts of the earlier waves
  {
    const int d = tid;
    int run = offsets[static_cast<int64_t>(d) * n_tiles + blockIdx.x];
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
      if (pos >= 0 && pos < n) {  // always true for consistent counts; keeps every store in bounds
        keys_out[pos] = key[bt];
        vals_out[pos] = vals_in ? vals_in[idx] : static_cast<int>(idx);
      }
    }
    // every leader has read its digit's start above; now advance it
    if (dig[bt] >= 0 && (__ffsll(static_cast<long long>(peer[bt])) - 1) == lane) wh[w][dig[bt]] += __popcll(peer[bt]);
  }
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

// seg[k] = first position whose code is >= k, k = 0..K
__global__ __launch_bounds__(256) void segment_bounds(const int* __restrict__ sorted_keys, const int* __restrict__ n_dev,
                                                      int64_t K, int* __restrict__ seg) {
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (k > K) return;
  int lo = 0, hi = *n_dev;
  while (lo < hi) {
    const int mid = lo + ((hi - lo) >> 1);
    if (sorted_keys[mid] < k)
      lo = mid + 1;
    else
      hi = mid;
  }
  seg[k] = lo;
}

__device__ __forceinline__ void store_centroid(void* C, int ct, int64_t k, int d, int t, double v) {
  if (ct == ET_F32)
    static_cast<float*>(C)[k * d + t] = static_cast<float>(v);
  else
    static_cast<uint16_t*>(C)[k * d + t] = bf16_from_double(v);
}

// One wave per code: lanes stride the segment, then a fixed xor-butterfly (identical in every lane).
__global__ __launch_bounds__(256) void segment_mean_wave(RowSrc src, const int* __restrict__ vals,
                                                         const int* __restrict__ seg, int64_t K, void* C, int ct,
                                                         int32_t* __restrict__ counts) {
  const int lane = threadIdx.x & 63;
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (k >= K) return;
  const int d = src.d;
  const int s = seg[k], e = seg[k + 1];
  if (counts && lane == 0) counts[k] = e - s;
  if (e == s) return;
  double acc[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) acc[t] = 0.0;
  for (int p = s + lane; p < e; p += 64) {
    const int64_t off = row_offset(src, vals[p]);
#pragma unroll
    for (int t = 0; t < 16; ++t)
      if (t < d) acc[t] = acc[t] + row_elem(src, off, t);
  }
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    if (t < d) {
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) acc[t] = acc[t] + __shfl_xor(acc[t], m);
    }
  }
  const double cnt = static_cast<double>(e - s);
#pragma unroll
  for (int t = 0; t < 16; ++t)
    if (t < d && lane == t) store_centroid(C, ct, k, d, t, acc[t] / cnt);
}

// One block per code for large segments: per-thread strided sums, then a fixed LDS tree.
__global__ __launch_bounds__(256) void segment_mean_block(RowSrc src, const int* __restrict__ vals,
                                                          const int* __restrict__ seg, int64_t K, void* C, int ct,
                                                          int32_t* __restrict__ counts) {
  __shared__ double sh[256 * 16];
  const int tid = threadIdx.x;
  const int64_t k = blockIdx.x;
  const int d = src.d;
  const int s = seg[k], e = seg[k + 1];
  if (counts && tid == 0) counts[k] = e - s;
  if (e == s) return;  // uniform across the block
  double acc[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) acc[t] = 0.0;
  for (int p = s + tid; p < e; p += 256) {
    const int64_t off = row_offset(src, vals[p]);
#pragma unroll
    for (int t = 0; t < 16; ++t)
      if (t < d) acc[t] = acc[t] + row_elem(src, off, t);
  }
#pragma unroll
  for (int t = 0; t < 16; ++t) sh[t * 256 + tid] = acc[t];
  __syncthreads();
  for (int stride = 128; stride >= 1; stride >>= 1) {
    if (tid < stride) {
#pragma unroll
      for (int t = 0; t < 16; ++t)
        if (t < d) sh[t * 256 + tid] = sh[t * 256 + tid] + sh[t * 256 + tid + stride];
    }
    __syncthreads();
  }
  if (tid < d) store_centroid(C, ct, k, d, tid, sh[tid * 256] / static_cast<double>(e - s));
}

// ---- small codebooks (K <= 256): one thread per code, no global sort --------------------------
// Each block walks a contiguous range of vectors in rounds of 2048.  A round's codes are stably
// bucket-sorted in LDS (the same ballot multisplit as the radix passes, so no atomics), then
// thread k adds the members of code k in ascending order to its fp64 accumulators.  The per-block
// partial sums are folded in block order by a second kernel.
constexpr int kRound = 2048;  // 4 waves x 8 batches x 64 lanes

__global__ __launch_bounds__(256) void small_k_partial(RowSrc src, const int32_t* __restrict__ codes, int64_t K,
                                                       int64_t per_block, double* __restrict__ part,
                                                       int* __restrict__ pcount) {
  __shared__ int s_pos[kRound];
  __shared__ int s_start[257];
  __shared__ int wh[4][256];
  __shared__ int sh_scan[256];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int d = src.d;
  const int64_t n = src.n;
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per_block;
  const int64_t b1 = (b0 + per_block < n) ? b0 + per_block : n;
  double acc[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) acc[t] = 0.0;
  int cnt = 0;
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int64_t base = b0; base < b1; base += kRound) {
    for (int b = tid; b < 1024; b += 256) (&wh[0][0])[b] = 0;
    __syncthreads();
    int dig[8];
    uint64_t peer[8];
#pragma unroll
    for (int bt = 0; bt < 8; ++bt) {
      const int64_t idx = base + w * 512 + bt * 64 + lane;
      const int c = (idx < b1) ? codes[idx] : -1;
      const bool valid = c >= 0 && c < K;
      dig[bt] = valid ? c : -1;
      peer[bt] = peer_mask(valid, valid ? c : 0);
      if (valid && (__ffsll(static_cast<long long>(peer[bt])) - 1) == lane) wh[w][c] += __popcll(peer[bt]);
    }
    __syncthreads();
    // bucket starts: exclusive scan over codes of the round's per-code totals
    const int tot = wh[0][tid] + wh[1][tid] + wh[2][tid] + wh[3][tid];
    sh_scan[tid] = tot;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
      const int v = (tid >= off) ? sh_scan[tid - off] : 0;
      __syncthreads();
      sh_scan[tid] += v;
      __syncthreads();
    }
    const int start = sh_scan[tid] - tot;
    s_start[tid] = start;
    if (tid == 255) s_start[256] = sh_scan[255];
    int run = start;
    for (int ww = 0; ww < 4; ++ww) {
      const int c = wh[ww][tid];
      wh[ww][tid] = run;
      run += c;
    }
    __syncthreads();
#pragma unroll
    for (int bt = 0; bt < 8; ++bt) {
      if (dig[bt] >= 0) {
        const int pos = wh[w][dig[bt]] + __popcll(peer[bt] & lt);
        if (pos >= 0 && pos < kRound) s_pos[pos] = w * 512 + bt * 64 + lane;
      }
      if (dig[bt] >= 0 && (__ffsll(static_cast<long long>(peer[bt])) - 1) == lane) wh[w][dig[bt]] += __popcll(peer[bt]);
    }
    __syncthreads();
    if (tid < K) {
      const int e = s_start[tid + 1];
      for (int j = s_start[tid]; j < e; ++j) {
        const int64_t off = row_offset(src, base + s_pos[j]);
#pragma unroll
        for (int t = 0; t < 16; ++t)
          if (t < d) acc[t] = acc[t] + row_elem(src, off, t);
      }
      cnt += e - s_start[tid];
    }
    __syncthreads();
  }
  if (tid < K) {
    double* pp = part + (static_cast<int64_t>(blockIdx.x) * K + tid) * d;
#pragma unroll
    for (int t = 0; t < 16; ++t)
      if (t < d) pp[t] = acc[t];
    pcount[static_cast<int64_t>(blockIdx.x) * K + tid] = cnt;
  }
}

__global__ __launch_bounds__(256) void small_k_final(const double* __restrict__ part, const int* __restrict__ pcount,
                                                     int blocks, int64_t K, int d, void* C, int ct,
                                                     int32_t* __restrict__ counts) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= K * d) return;
  const int64_t k = e / d;
  const int t = static_cast<int>(e - k * d);
  double acc = 0.0;
  int cnt = 0;
  for (int b = 0; b < blocks; ++b) {
    acc = acc + part[(static_cast<int64_t>(b) * K + k) * d + t];
    cnt += pcount[static_cast<int64_t>(b) * K + k];
  }
  if (counts && t == 0) counts[k] = cnt;
  if (cnt > 0) store_centroid(C, ct, k, d, t, acc / static_cast<double>(cnt));
}

struct SmallPlan {
  int64_t blocks;
  int64_t per_block;
};

SmallPlan small_plan(int64_t n) {
  SmallPlan p;
  const int64_t rounds = cdiv(n > 0 ? n : 1, kRound);
  p.blocks = rounds < 512 ? rounds : 512;
  p.per_block = cdiv(rounds, p.blocks) * kRound;
  p.blocks = cdiv(n > 0 ? n : 1, p.per_block);
  return p;
}

struct KmWs {
  int* keys[2];
  int* vals[2];
  int* hist;
  int* offs;
  int* sums;
  int* n_valid;
  int* seg;
};

KmWs carve(WsCursor& ws, int64_t n, int64_t K) {
  KmWs w;
  const int64_t n_tiles = cdiv(n > 0 ? n : 1, kTile);
  const int64_t hn = 256 * n_tiles;
  for (int b = 0; b < 2; ++b) {
    w.keys[b] = ws.take<int>(static_cast<size_t>(n));
    w.vals[b] = ws.take<int>(static_cast<size_t>(n));
  }
  w.hist = ws.take<int>(static_cast<size_t>(hn));
  w.offs = ws.take<int>(static_cast<size_t>(hn));
  w.sums = ws.take<int>(static_cast<size_t>(cdiv(hn, kScanBlock)));
  w.n_valid = ws.take<int>(1);
  w.seg = ws.take<int>(static_cast<size_t>(K + 1));
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
    SmallPlan p = small_plan(n);
    c.take<double>(static_cast<size_t>(p.blocks * K * 16));
    c.take<int>(static_cast<size_t>(p.blocks * K));
    return c.used;
  }
  carve(c, n, K);
  return c.used;
}

hipError_t launch_kmeans_update(const RowSrc& src, const int32_t* codes, int64_t K, void* C, int c_type,
                                int32_t* counts, void* ws, hipStream_t stream) {
  const int64_t n = src.n;
  WsCursor cur(ws);
  if (K <= 256) {
    SmallPlan p = small_plan(n);
    double* part = cur.take<double>(static_cast<size_t>(p.blocks * K * 16));
    int* pcount = cur.take<int>(static_cast<size_t>(p.blocks * K));
    hipLaunchKernelGGL(small_k_partial, dim3(static_cast<unsigned>(p.blocks)), dim3(256), 0, stream, src, codes, K,
                       p.per_block, part, pcount);
    hipLaunchKernelGGL(small_k_final, dim3(static_cast<unsigned>(cdiv(K * src.d, 256))), dim3(256), 0, stream, part,
                       pcount, static_cast<int>(p.blocks), K, src.d, C, c_type, counts);
    return hipGetLastError();
  }
  KmWs w = carve(cur, n, K);
  const int64_t n_tiles = cdiv(n > 0 ? n : 1, kTile);
  const int passes = (K <= 256) ? 1 : 2;
  const int* kin = codes;
  const int* vin = nullptr;
  hipError_t e;
  for (int p = 0; p < passes; ++p) {
    const int* ndev = (p == 0) ? nullptr : w.n_valid;
    hipLaunchKernelGGL(radix_hist, dim3(static_cast<unsigned>(n_tiles)), dim3(256), 0, stream, kin, ndev, n, K, p, 8 * p,
                       n_tiles, w.hist);
    if ((e = exclusive_scan(w.hist, 256 * n_tiles, w.sums, w.offs, p == 0 ? w.n_valid : nullptr, stream)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(radix_scatter, dim3(static_cast<unsigned>(n_tiles)), dim3(256), 0, stream, kin, vin, ndev, n, K, p,
                       8 * p, n_tiles, w.offs, w.keys[p & 1], w.vals[p & 1]);
    kin = w.keys[p & 1];
    vin = w.vals[p & 1];
  }
  hipLaunchKernelGGL(segment_bounds, dim3(static_cast<unsigned>(cdiv(K + 1, 256))), dim3(256), 0, stream, kin,
                     w.n_valid, K, w.seg);
  if (n >= 256 * K) {
    hipLaunchKernelGGL(segment_mean_block, dim3(static_cast<unsigned>(K)), dim3(256), 0, stream, src, vin, w.seg, K, C,
                       c_type, counts);
  } else {
    hipLaunchKernelGGL(segment_mean_wave, dim3(static_cast<unsigned>(cdiv(K, 4))), dim3(256), 0, stream, src, vin, w.seg,
                       K, C, c_type, counts);
  }
  return hipGetLastError();
}

}  // namespace crvq
