// Host side of the libcrvq C ABI: argument validation (before anything is enqueued), workspace
// sizing, and dispatch to the kernel launchers.  See include/crvq.h for the contract of each call.
#include "crvq.h"
#include <cmath>

#include "crvq_internal.h"

#include <rocprofiler-sdk-roctx/roctx.h>

#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

using namespace crvq;

// Scratch of crvq_assign_noalloc: one array per GPU in the library's own device memory, kept until
// the process ends.  In host code `scratch` names a host-side stand-in, never the device array: its
// device address comes from hipGetSymbolAddress, once per device (scratch_on_device below).
static __device__ __align__(256) unsigned char scratch[CRVQ_NOALLOC_SCRATCH_BYTES];

namespace {

// A profiler range named after the entry point around each call that enqueues device work (seen by
// rocprofv3 --marker-trace; a function call and a check when no profiler is attached).
struct ApiRange {
  explicit ApiRange(const char* name) { roctxRangePushA(name); }
  ~ApiRange() { roctxRangePop(); }
  ApiRange(const ApiRange&) = delete;
  ApiRange& operator=(const ApiRange&) = delete;
};

thread_local std::string g_err;

crvq_status fail(crvq_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

crvq_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return CRVQ_OK;
  return fail(CRVQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool dtype_ok(int t) { return t == CRVQ_F32 || t == CRVQ_BF16; }
int esize(int t) { return t == CRVQ_F32 ? 4 : 2; }

crvq_status check_vectors(const void* X, int dtype, int64_t n_rows, int64_t vpr, int64_t ld, int32_t d,
                          const char* fn) {
  if (!dtype_ok(dtype)) return fail(CRVQ_ERR_INVALID, "%s: x_dtype %d is not CRVQ_F32 or CRVQ_BF16", fn, dtype);
  if (d < 1 || d > CRVQ_MAX_D) return fail(CRVQ_ERR_UNSUPPORTED, "%s: d = %d outside [1, %d]", fn, d, CRVQ_MAX_D);
  if (n_rows < 0 || vpr < 0) return fail(CRVQ_ERR_INVALID, "%s: negative n_rows or vecs_per_row", fn);
  if (ld < vpr * d) return fail(CRVQ_ERR_INVALID, "%s: ld = %lld < vecs_per_row * d = %lld", fn, (long long)ld,
                                (long long)(vpr * d));
  const int64_t n = n_rows * vpr;
  if (n > 0x7fffffffLL) return fail(CRVQ_ERR_UNSUPPORTED, "%s: %lld vectors exceed 2^31 - 1", fn, (long long)n);
  if (n > 0 && !X) return fail(CRVQ_ERR_INVALID, "%s: X is NULL", fn);
  return CRVQ_OK;
}

crvq_status check_K(int64_t K, const char* fn, const char* what) {
  if (K < 1 || K > CRVQ_MAX_K) return fail(CRVQ_ERR_INVALID, "%s: %s = %lld outside [1, %d]", fn, what, (long long)K, CRVQ_MAX_K);
  return CRVQ_OK;
}

crvq_status check_ws(void* ws, size_t have, size_t need, const char* fn) {
  if (need == 0) return CRVQ_OK;
  if (!ws || have < need)
    return fail(CRVQ_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given%s", fn, need, ws ? have : 0,
                ws ? "" : " (NULL)");
  if (reinterpret_cast<uintptr_t>(ws) & 255) return fail(CRVQ_ERR_WORKSPACE, "%s: workspace is not 256-byte aligned", fn);
  return CRVQ_OK;
}

RowSrc vec_src(const void* X, int dtype, int64_t n_rows, int64_t vpr, int64_t ld, int32_t d) {
  RowSrc s;
  s.base = X;
  s.type = dtype;
  s.d = d;
  s.vpr = vpr > 0 ? vpr : 1;
  s.ld = ld;
  s.n = n_rows * vpr;
  return s;
}

size_t assign_ws(int64_t n, int32_t d, int64_t K) {
  WsCursor c(nullptr);
  ScreenPlan p = plan_screen(n, d, K, 1);
  carve_screen(c, p, n, K);
  return c.used;
}

size_t beam_screen_bytes(int64_t n, int32_t d, int32_t n_books, const int64_t* Ks, int32_t beam) {
  size_t mx = 0;
  int64_t n_par = 1;
  for (int t = 0; t < n_books; ++t) {
    WsCursor c(nullptr);
    const int64_t rows = n * n_par;
    ScreenPlan p = plan_screen(rows, d, Ks[t], beam);
    carve_screen(c, p, rows, Ks[t]);
    if (c.used > mx) mx = c.used;
    const int64_t nn = n_par * Ks[t];
    n_par = nn < beam ? nn : beam;
  }
  return mx;
}

struct BeamWs {
  double* res[2];
  int* tup[2];
  double* err;
  double* rowD;
  int* rowK;
  char* screen;
};

BeamWs carve_beam(WsCursor& c, int64_t n, int32_t d, int32_t n_books, int32_t beam, size_t screen_bytes) {
  BeamWs w;
  const size_t nb = static_cast<size_t>(n) * beam;
  for (int b = 0; b < 2; ++b) {
    w.res[b] = c.take<double>(nb * d);
    w.tup[b] = c.take<int>(nb * n_books);
  }
  w.err = c.take<double>(nb);
  w.rowD = c.take<double>(nb * beam);
  w.rowK = c.take<int>(nb * beam);
  w.screen = c.take<char>(screen_bytes);
  return w;
}

bool overlaps(const void* a, size_t an, const void* b, size_t bn) {
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  return pa < pb + bn && pb < pa + an;
}

}  // namespace

extern "C" {

int crvq_version(void) { return 100; }

const char* crvq_last_error(void) { return g_err.c_str(); }

// ------------------------------------------------------------------------------------------------
size_t crvq_importance_workspace_size(int64_t M, int64_t N) {
  if (M < 1 || N < 1) return 0;
  return colreduce_ws_bytes(M, N);
}

crvq_status crvq_channel_importance(const void* A, int64_t lda, const void* B, int64_t ldb, int dtype, int64_t M,
                                    int64_t N, const float* scale, int reduce, float* out, void* workspace,
                                    size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_channel_importance");
  static const char* fn = "crvq_channel_importance";
  g_err.clear();
  if (!dtype_ok(dtype)) return fail(CRVQ_ERR_INVALID, "%s: dtype %d is not CRVQ_F32 or CRVQ_BF16", fn, dtype);
  if (M < 1 || N < 1) return fail(CRVQ_ERR_INVALID, "%s: M and N must be >= 1 (got %lld, %lld)", fn, (long long)M, (long long)N);
  if (!A || !out) return fail(CRVQ_ERR_INVALID, "%s: A and out must not be NULL", fn);
  if (lda < N) return fail(CRVQ_ERR_INVALID, "%s: lda < N", fn);
  if (B && ldb < N) return fail(CRVQ_ERR_INVALID, "%s: ldb < N", fn);
  if (reduce != CRVQ_REDUCE_SUM && reduce != CRVQ_REDUCE_MAX) return fail(CRVQ_ERR_INVALID, "%s: unknown reduce %d", fn, reduce);
  crvq_status s = check_ws(workspace, ws_bytes, colreduce_ws_bytes(M, N), fn);
  if (s) return s;
  return hip_status(launch_colreduce(A, lda, B, ldb, dtype, M, N, scale, reduce, out, workspace,
                                     static_cast<hipStream_t>(stream)),
                    fn);
}

// ------------------------------------------------------------------------------------------------
size_t crvq_reorder_workspace_size(int64_t N) {
  if (N < 1) return 0;
  return align256(static_cast<size_t>(N) * 4) + align256(static_cast<size_t>(rank_chunks(N)) * N * 4);
}

crvq_status crvq_reorder(const void* in, int64_t ld_in, void* out, int64_t ld_out, int dtype, int64_t M, int64_t N,
                         const float* importance, int32_t* perm, int inverse, void* workspace, size_t ws_bytes,
                         void* stream) {
  const ApiRange range("crvq_reorder");
  static const char* fn = "crvq_reorder";
  g_err.clear();
  if (N < 1 || N > (1LL << 20)) return fail(CRVQ_ERR_INVALID, "%s: N = %lld outside [1, 2^20]", fn, (long long)N);
  if (!perm) return fail(CRVQ_ERR_INVALID, "%s: perm must not be NULL", fn);
  if (!importance && !in) return fail(CRVQ_ERR_INVALID, "%s: nothing to do (importance and in are both NULL)", fn);
  if (in) {
    if (!dtype_ok(dtype)) return fail(CRVQ_ERR_INVALID, "%s: dtype %d is not CRVQ_F32 or CRVQ_BF16", fn, dtype);
    if (M < 0) return fail(CRVQ_ERR_INVALID, "%s: M < 0", fn);
    if (!out) return fail(CRVQ_ERR_INVALID, "%s: out must not be NULL", fn);
    if (ld_in < N || ld_out < N) return fail(CRVQ_ERR_INVALID, "%s: ld_in and ld_out must be >= N", fn);
    if (M > 0) {
      const size_t es = esize(dtype);
      const size_t span_in = static_cast<size_t>((M - 1) * ld_in + N) * es;
      const size_t span_out = static_cast<size_t>((M - 1) * ld_out + N) * es;
      if (overlaps(in, span_in, out, span_out)) return fail(CRVQ_ERR_INVALID, "%s: in and out overlap", fn);
    }
  }
  if (importance || (in && inverse)) {
    crvq_status s = check_ws(workspace, ws_bytes, crvq_reorder_workspace_size(N), fn);
    if (s) return s;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t* inv_ws = static_cast<int32_t*>(workspace);
  int32_t* rank_ws = inv_ws ? inv_ws + align256(static_cast<size_t>(N) * 4) / 4 : nullptr;
  if (importance) {
    crvq_status s = hip_status(launch_rank_perm(importance, N, perm, rank_ws, st), fn);
    if (s) return s;
  }
  if (!in || M == 0) return CRVQ_OK;
  const int32_t* src = perm;
  if (inverse) {
    crvq_status s = hip_status(launch_inverse_perm(perm, N, inv_ws, st), fn);
    if (s) return s;
    src = inv_ws;
  }
  return hip_status(launch_gather_columns(in, ld_in, out, ld_out, esize(dtype), M, N, src, st), fn);
}

// ------------------------------------------------------------------------------------------------
size_t crvq_assign_workspace_size(int64_t n_vectors, int32_t d, int64_t K) {
  if (n_vectors < 1 || d < 1 || d > CRVQ_MAX_D || K < 1 || K > CRVQ_MAX_K) return 0;
  return assign_ws(n_vectors, d, K);
}

crvq_status crvq_assign(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld, int32_t d,
                        const void* C, int c_dtype, int64_t K, int32_t* codes, float* dist, void* workspace,
                        size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_assign");
  static const char* fn = "crvq_assign";
  g_err.clear();
  crvq_status s = check_vectors(X, x_dtype, n_rows, vecs_per_row, ld, d, fn);
  if (s) return s;
  if (!dtype_ok(c_dtype)) return fail(CRVQ_ERR_INVALID, "%s: c_dtype %d is not CRVQ_F32 or CRVQ_BF16", fn, c_dtype);
  if ((s = check_K(K, fn, "K"))) return s;
  if (!C) return fail(CRVQ_ERR_INVALID, "%s: C must not be NULL", fn);
  const int64_t n = n_rows * vecs_per_row;
  if (n > 0 && !codes) return fail(CRVQ_ERR_INVALID, "%s: codes must not be NULL", fn);
  if (n == 0) return CRVQ_OK;
  if ((s = check_ws(workspace, ws_bytes, assign_ws(n, d, K), fn))) return s;
  RowSrc src = vec_src(X, x_dtype, n_rows, vecs_per_row, ld, d);
  ScreenPlan p = plan_screen(n, d, K, 1);
  WsCursor c(workspace);
  ScreenWs w = carve_screen(c, p, n, K);
  return hip_status(launch_screen(src, C, c_dtype, K, 1, p, w, codes, dist, nullptr, nullptr,
                                  static_cast<hipStream_t>(stream)),
                    fn);
}

// ------------------------------------------------------------------------------------------------
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// The device address of `scratch` on the current device (looked up on the first call there).
crvq_status scratch_on_device(void** out, const char* fn) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, fn);
  if (dev < 0 || dev >= kMaxDevices) return fail(CRVQ_ERR_UNSUPPORTED, "%s: device %d beyond %d", fn, dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, fn);
    if (!p) return fail(CRVQ_ERR_HIP, "%s: no device address for the scratch array on device %d", fn, dev);
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return CRVQ_OK;
}

}  // namespace

crvq_status crvq_assign_noalloc(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld,
                                int32_t d, const void* C, int c_dtype, int64_t K, int32_t* codes, float* dist,
                                void* stream) {
  const ApiRange range("crvq_assign_noalloc");
  static const char* fn = "crvq_assign_noalloc";
  g_err.clear();
  crvq_status s = check_vectors(X, x_dtype, n_rows, vecs_per_row, ld, d, fn);
  if (s) return s;
  if (!dtype_ok(c_dtype)) return fail(CRVQ_ERR_INVALID, "%s: c_dtype %d is not CRVQ_F32 or CRVQ_BF16", fn, c_dtype);
  if ((s = check_K(K, fn, "K"))) return s;
  if (!C) return fail(CRVQ_ERR_INVALID, "%s: C must not be NULL", fn);
  const int64_t n = n_rows * vecs_per_row;
  if (n > 0 && !codes) return fail(CRVQ_ERR_INVALID, "%s: codes must not be NULL", fn);
  if (n == 0) return CRVQ_OK;
  const size_t need = assign_ws(n, d, K);
  if (need > static_cast<size_t>(CRVQ_NOALLOC_SCRATCH_BYTES))
    return fail(CRVQ_ERR_UNSUPPORTED, "%s: %lld vectors against %lld codewords need %zu bytes of scratch, beyond the "
                "fixed %lld (use crvq_assign with a workspace)", fn, (long long)n, (long long)K, need,
                (long long)CRVQ_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((s = scratch_on_device(&ws, fn))) return s;
  RowSrc src = vec_src(X, x_dtype, n_rows, vecs_per_row, ld, d);
  ScreenPlan p = plan_screen(n, d, K, 1);
  WsCursor c(ws);
  ScreenWs w = carve_screen(c, p, n, K);
  return hip_status(launch_screen(src, C, c_dtype, K, 1, p, w, codes, dist, nullptr, nullptr,
                                  static_cast<hipStream_t>(stream)),
                    fn);
}

// ------------------------------------------------------------------------------------------------
size_t crvq_beam_workspace_size(int64_t n_vectors, int32_t d, int32_t n_books, const int64_t* Ks, int32_t beam) {
  if (n_vectors < 1 || d < 1 || d > CRVQ_MAX_D || n_books < 1 || n_books > CRVQ_MAX_BOOKS || !Ks || beam < 1 ||
      beam > CRVQ_MAX_BEAM)
    return 0;
  for (int t = 0; t < n_books; ++t)
    if (Ks[t] < 1 || Ks[t] > CRVQ_MAX_K) return 0;
  const size_t sb = beam_screen_bytes(n_vectors, d, n_books, Ks, beam);
  WsCursor c(nullptr);
  carve_beam(c, n_vectors, d, n_books, beam, sb);
  return c.used;
}

crvq_status crvq_assign_residual_beam(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld,
                                      int32_t d, int32_t n_books, const void* const* books, const int32_t* book_dtypes,
                                      const int64_t* Ks, int32_t beam, int32_t* const* codes, const int64_t* ldc,
                                      float* err, void* workspace, size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_assign_residual_beam");
  static const char* fn = "crvq_assign_residual_beam";
  g_err.clear();
  crvq_status s = check_vectors(X, x_dtype, n_rows, vecs_per_row, ld, d, fn);
  if (s) return s;
  if (n_books < 1 || n_books > CRVQ_MAX_BOOKS)
    return fail(CRVQ_ERR_INVALID, "%s: n_books = %d outside [1, %d]", fn, n_books, CRVQ_MAX_BOOKS);
  if (beam < 1 || beam > CRVQ_MAX_BEAM) return fail(CRVQ_ERR_INVALID, "%s: beam = %d outside [1, %d]", fn, beam, CRVQ_MAX_BEAM);
  if (!books || !book_dtypes || !Ks || !codes) return fail(CRVQ_ERR_INVALID, "%s: books, book_dtypes, Ks and codes must not be NULL", fn);
  for (int t = 0; t < n_books; ++t) {
    if (!books[t] || !codes[t]) return fail(CRVQ_ERR_INVALID, "%s: books[%d] or codes[%d] is NULL", fn, t, t);
    if (!dtype_ok(book_dtypes[t])) return fail(CRVQ_ERR_INVALID, "%s: book_dtypes[%d] = %d invalid", fn, t, book_dtypes[t]);
    if ((s = check_K(Ks[t], fn, "Ks[t]"))) return s;
    if (ldc && ldc[t] < vecs_per_row) return fail(CRVQ_ERR_INVALID, "%s: ldc[%d] < vecs_per_row", fn, t);
  }
  const int64_t n = n_rows * vecs_per_row;
  if (n == 0) return CRVQ_OK;
  const size_t sb = beam_screen_bytes(n, d, n_books, Ks, beam);
  {
    WsCursor dry(nullptr);
    carve_beam(dry, n, d, n_books, beam, sb);
    if ((s = check_ws(workspace, ws_bytes, dry.used, fn))) return s;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  WsCursor c(workspace);
  BeamWs w = carve_beam(c, n, d, n_books, beam, sb);
  const RowSrc src0 = vec_src(X, x_dtype, n_rows, vecs_per_row, ld, d);
  int64_t n_par = 1;
  int cur = 0;
  for (int t = 0; t < n_books; ++t) {
    const int64_t rows = n * n_par;
    RowSrc src = src0;
    if (t > 0) {
      src.base = w.res[cur];
      src.type = ET_F64;
      src.vpr = 1;
      src.ld = d;
      src.n = rows;
    }
    ScreenPlan p = plan_screen(rows, d, Ks[t], beam);
    WsCursor sc(w.screen);
    ScreenWs sw = carve_screen(sc, p, rows, Ks[t]);
    hipError_t e = launch_screen(src, books[t], book_dtypes[t], Ks[t], beam, p, sw, nullptr, nullptr, w.rowD, w.rowK, st);
    if (e != hipSuccess) return hip_status(e, fn);
    e = launch_beam_merge(n, static_cast<int>(n_par), beam, t, n_books, w.rowD, w.rowK, src0, w.res[cur], w.res[cur ^ 1],
                          w.tup[cur], w.tup[cur ^ 1], w.err, books[t], book_dtypes[t], Ks[t], d, st);
    if (e != hipSuccess) return hip_status(e, fn);
    const int64_t nn = n_par * Ks[t];
    n_par = nn < beam ? nn : beam;
    cur ^= 1;
  }
  CodePtrs outs = {};
  for (int t = 0; t < n_books; ++t) {
    outs.q[t] = codes[t];
    outs.ld[t] = ldc ? ldc[t] : vecs_per_row;
  }
  return hip_status(launch_beam_emit(n, vecs_per_row, static_cast<int>(n_par), n_books, w.tup[cur], w.err, outs, err, st),
                    fn);
}

// ------------------------------------------------------------------------------------------------
size_t crvq_kmeans_workspace_size(int64_t n_vectors, int32_t d, int64_t K) {
  (void)d;
  if (n_vectors < 0 || K < 1 || K > CRVQ_MAX_K) return 0;
  return kmeans_ws_bytes(n_vectors, K);
}

crvq_status crvq_kmeans_update(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld, int32_t d,
                               const int32_t* codes, int64_t K, void* C, int c_dtype, int32_t* counts, void* workspace,
                               size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_kmeans_update");
  static const char* fn = "crvq_kmeans_update";
  g_err.clear();
  crvq_status s = check_vectors(X, x_dtype, n_rows, vecs_per_row, ld, d, fn);
  if (s) return s;
  if ((s = check_K(K, fn, "K"))) return s;
  if (!C) return fail(CRVQ_ERR_INVALID, "%s: C must not be NULL", fn);
  if (!dtype_ok(c_dtype)) return fail(CRVQ_ERR_INVALID, "%s: c_dtype %d is not CRVQ_F32 or CRVQ_BF16", fn, c_dtype);
  const int64_t n = n_rows * vecs_per_row;
  if (n > 0 && !codes) return fail(CRVQ_ERR_INVALID, "%s: codes must not be NULL", fn);
  if ((s = check_ws(workspace, ws_bytes, kmeans_ws_bytes(n, K), fn))) return s;
  return hip_status(launch_kmeans_update(vec_src(X, x_dtype, n_rows, vecs_per_row, ld, d), codes, K, C, c_dtype, counts,
                                         workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

// ------------------------------------------------------------------------------------------------
crvq_status crvq_gather_vectors(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld,
                                int32_t d, const int64_t* idx, int64_t count, void* out, int out_dtype, void* stream) {
  const ApiRange range("crvq_gather_vectors");
  static const char* fn = "crvq_gather_vectors";
  g_err.clear();
  crvq_status s = check_vectors(X, x_dtype, n_rows, vecs_per_row, ld, d, fn);
  if (s) return s;
  if (count < 0) return fail(CRVQ_ERR_INVALID, "%s: count < 0", fn);
  if (out_dtype != x_dtype && !(x_dtype == CRVQ_BF16 && out_dtype == CRVQ_F32))
    return fail(CRVQ_ERR_INVALID, "%s: out_dtype must equal x_dtype (or be F32 for BF16 input)", fn);
  if (count == 0) return CRVQ_OK;
  if (!idx || !out) return fail(CRVQ_ERR_INVALID, "%s: idx and out must not be NULL", fn);
  return hip_status(launch_gather_vectors(vec_src(X, x_dtype, n_rows, vecs_per_row, ld, d), idx, count, out, out_dtype,
                                          static_cast<hipStream_t>(stream)),
                    fn);
}

// ------------------------------------------------------------------------------------------------
size_t crvq_dequant_workspace_size(int64_t n_cols) { return n_cols < 1 ? 0 : align256(static_cast<size_t>(n_cols) * 4); }

// Shared by crvq_dequant (one basic book) and crvq_dequant_books (n_base of them): books[0, n_base)
// cover every vector with code stride ldq_base, books[n_base, n_base + n_ext) the critical groups with
// stride ldq_ext.
static crvq_status dequant_impl(const char* fn, int64_t M, int64_t n_cols, int32_t d, int64_t n_crit, int32_t n_base,
                                int32_t n_ext, const int32_t* const* q, int64_t ldq_base, int64_t ldq_ext,
                                const void* const* C, const int32_t* dtypes, const int64_t* Ks, const int32_t* perm,
                                const void* minuend, int minuend_dtype, int64_t ld_min, void* out, int out_dtype,
                                int64_t ld_out, void* workspace, size_t ws_bytes, void* stream) {
  g_err.clear();
  if (M < 0 || n_cols < 1) return fail(CRVQ_ERR_INVALID, "%s: need M >= 0 and n_cols >= 1", fn);
  if (d < 1 || d > CRVQ_MAX_D) return fail(CRVQ_ERR_UNSUPPORTED, "%s: d = %d outside [1, %d]", fn, d, CRVQ_MAX_D);
  if (n_cols % d) return fail(CRVQ_ERR_INVALID, "%s: n_cols = %lld is not a multiple of d = %d", fn, (long long)n_cols, d);
  if (n_crit < 0 || n_crit > n_cols || n_crit % d)
    return fail(CRVQ_ERR_INVALID, "%s: n_crit = %lld must be a multiple of d in [0, n_cols]", fn, (long long)n_crit);
  if (n_base < 1 || n_ext < 0 || n_base + n_ext > CRVQ_MAX_BOOKS)
    return fail(CRVQ_ERR_INVALID, "%s: need n_base >= 1, n_ext >= 0 and n_base + n_ext <= %d (got %d + %d)", fn,
                CRVQ_MAX_BOOKS, n_base, n_ext);
  if (!out) return fail(CRVQ_ERR_INVALID, "%s: out must not be NULL", fn);
  if (!dtype_ok(out_dtype) && !(out_dtype == CRVQ_F64 && !perm))
    return fail(CRVQ_ERR_INVALID, "%s: invalid out dtype (CRVQ_F64 only without perm)", fn);
  if (ldq_base < n_cols / d) return fail(CRVQ_ERR_INVALID, "%s: ldq_base < n_cols / d", fn);
  if (n_ext > 0 && ldq_ext < n_crit / d) return fail(CRVQ_ERR_INVALID, "%s: ldq_ext < n_crit / d", fn);
  if (ld_out < n_cols) return fail(CRVQ_ERR_INVALID, "%s: ld_out < n_cols", fn);
  if (perm && minuend) return fail(CRVQ_ERR_INVALID, "%s: perm and minuend are mutually exclusive", fn);
  if (minuend) {
    if (!dtype_ok(minuend_dtype)) return fail(CRVQ_ERR_INVALID, "%s: invalid minuend dtype", fn);
    if (ld_min < n_cols) return fail(CRVQ_ERR_INVALID, "%s: ld_min < n_cols", fn);
  }
  DequantBooks b = {};
  b.n = n_base + n_ext;
  b.n_full = n_base;
  b.ldq_base = ldq_base;
  b.ldq_ext = ldq_ext;
  crvq_status s = CRVQ_OK;
  for (int e = 0; e < b.n; ++e) {
    if (!q[e] || !C[e]) return fail(CRVQ_ERR_INVALID, "%s: the code array or codebook of book %d is NULL", fn, e);
    if (!dtype_ok(dtypes[e])) return fail(CRVQ_ERR_INVALID, "%s: the dtype of book %d is invalid", fn, e);
    if ((s = check_K(Ks[e], fn, "K"))) return s;
    b.C[e] = C[e];
    b.q[e] = q[e];
    b.type[e] = dtypes[e];
    b.K[e] = Ks[e];
  }
  if (perm && (s = check_ws(workspace, ws_bytes, crvq_dequant_workspace_size(n_cols), fn))) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t* inv = nullptr;
  if (perm) {
    inv = static_cast<int32_t*>(workspace);
    if ((s = hip_status(launch_inverse_perm(perm, n_cols, inv, st), fn))) return s;
  }
  return hip_status(
      launch_dequant(M, n_cols, d, n_crit, b, inv, perm, minuend, minuend_dtype, ld_min, out, out_dtype, ld_out, st), fn);
}

crvq_status crvq_dequant(int64_t M, int64_t n_cols, int32_t d, int64_t n_crit, const int32_t* q_base,
                         int64_t ldq_base, const void* C_base, int base_dtype, int64_t K_base, int32_t n_ext,
                         const int32_t* const* q_ext, int64_t ldq_ext, const void* const* C_ext,
                         const int32_t* ext_dtypes, const int64_t* K_ext, const int32_t* perm, const void* minuend,
                         int minuend_dtype, int64_t ld_min, void* out, int out_dtype, int64_t ld_out, void* workspace,
                         size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_dequant");
  static const char* fn = "crvq_dequant";
  g_err.clear();
  if (n_ext < 0 || n_ext > CRVQ_MAX_BOOKS - 1)
    return fail(CRVQ_ERR_INVALID, "%s: n_ext = %d outside [0, %d]", fn, n_ext, CRVQ_MAX_BOOKS - 1);
  if (!q_base || !C_base) return fail(CRVQ_ERR_INVALID, "%s: q_base and C_base must not be NULL", fn);
  if (n_ext > 0 && (!q_ext || !C_ext || !ext_dtypes || !K_ext))
    return fail(CRVQ_ERR_INVALID, "%s: q_ext, C_ext, ext_dtypes and K_ext must not be NULL when n_ext > 0", fn);
  const int32_t* q[CRVQ_MAX_BOOKS] = {q_base};
  const void* C[CRVQ_MAX_BOOKS] = {C_base};
  int32_t dts[CRVQ_MAX_BOOKS] = {base_dtype};
  int64_t Ks[CRVQ_MAX_BOOKS] = {K_base};
  for (int e = 0; e < n_ext; ++e) {
    q[e + 1] = q_ext[e];
    C[e + 1] = C_ext[e];
    dts[e + 1] = ext_dtypes[e];
    Ks[e + 1] = K_ext[e];
  }
  return dequant_impl(fn, M, n_cols, d, n_crit, 1, n_ext, q, ldq_base, ldq_ext, C, dts, Ks, perm, minuend, minuend_dtype,
                      ld_min, out, out_dtype, ld_out, workspace, ws_bytes, stream);
}

crvq_status crvq_dequant_books(int64_t M, int64_t n_cols, int32_t d, int64_t n_crit, int32_t n_base, int32_t n_ext,
                               const int32_t* const* q, int64_t ldq_base, int64_t ldq_ext, const void* const* C,
                               const int32_t* dtypes, const int64_t* Ks, const int32_t* perm, const void* minuend,
                               int minuend_dtype, int64_t ld_min, void* out, int out_dtype, int64_t ld_out,
                               void* workspace, size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_dequant_books");
  static const char* fn = "crvq_dequant_books";
  g_err.clear();
  if (!q || !C || !dtypes || !Ks) return fail(CRVQ_ERR_INVALID, "%s: q, C, dtypes and Ks must not be NULL", fn);
  return dequant_impl(fn, M, n_cols, d, n_crit, n_base, n_ext, q, ldq_base, ldq_ext, C, dtypes, Ks, perm, minuend,
                      minuend_dtype, ld_min, out, out_dtype, ld_out, workspace, ws_bytes, stream);
}

crvq_status crvq_bits_per_weight(int64_t rows, int64_t cols, int32_t d, int64_t n_crit, int32_t n_base, int32_t n_ext,
                                 const int64_t* Ks, int32_t codeword_bits, int32_t perm_bits, double* out) {
  static const char* fn = "crvq_bits_per_weight";
  g_err.clear();
  if (rows < 1 || cols < 1) return fail(CRVQ_ERR_INVALID, "%s: need rows >= 1 and cols >= 1", fn);
  if (d < 1 || d > CRVQ_MAX_D || cols % d) return fail(CRVQ_ERR_INVALID, "%s: d = %d must be in [1, %d] and divide cols", fn, d, CRVQ_MAX_D);
  if (n_crit < 0 || n_crit > cols || n_crit % d)
    return fail(CRVQ_ERR_INVALID, "%s: n_crit = %lld must be a multiple of d in [0, cols]", fn, (long long)n_crit);
  if (n_base < 1 || n_ext < 0 || n_base + n_ext > CRVQ_MAX_BOOKS)
    return fail(CRVQ_ERR_INVALID, "%s: need n_base >= 1, n_ext >= 0 and n_base + n_ext <= %d", fn, CRVQ_MAX_BOOKS);
  if (codeword_bits < 1 || codeword_bits > 64 || perm_bits < 0 || perm_bits > 64)
    return fail(CRVQ_ERR_INVALID, "%s: codeword_bits must be in [1, 64] and perm_bits in [0, 64]", fn);
  if (!Ks || !out) return fail(CRVQ_ERR_INVALID, "%s: Ks and out must not be NULL", fn);
  // every count below is an integer well inside 2^53, so the sums are exact in double
  const double full_vecs = static_cast<double>(rows) * static_cast<double>(cols / d);
  const double crit_vecs = static_cast<double>(rows) * static_cast<double>(n_crit / d);
  double bits = static_cast<double>(cols) * perm_bits;
  for (int b = 0; b < n_base + n_ext; ++b) {
    crvq_status s = check_K(Ks[b], fn, "Ks[b]");
    if (s) return s;
    int e = 0;
    while ((int64_t{1} << e) < Ks[b]) ++e;
    bits += (b < n_base ? full_vecs : crit_vecs) * e;
    bits += static_cast<double>(Ks[b]) * d * codeword_bits;
  }
  *out = bits / (static_cast<double>(rows) * static_cast<double>(cols));
  return CRVQ_OK;
}

// ---- loss-driven refinement ----------------------------------------------------------------------
crvq_status crvq_gram(const void* X, int x_dtype, int64_t n_rows, int64_t n_cols, int64_t ld, double* H, int64_t ldh,
                      void* stream) {
  const ApiRange range("crvq_gram");
  static const char* fn = "crvq_gram";
  g_err.clear();
  if (n_rows < 0 || n_cols < 0) return fail(CRVQ_ERR_INVALID, "%s: negative size", fn);
  if (x_dtype != CRVQ_F32 && x_dtype != CRVQ_F64) return fail(CRVQ_ERR_INVALID, "%s: x_dtype must be F32 or F64", fn);
  if (ld < n_cols || ldh < n_cols) return fail(CRVQ_ERR_INVALID, "%s: ld and ldh must be >= n_cols", fn);
  if (n_cols == 0) return CRVQ_OK;
  if (!H || (n_rows > 0 && !X)) return fail(CRVQ_ERR_INVALID, "%s: X and H must not be NULL", fn);
  return hip_status(launch_gemm_f64(n_cols, n_cols, n_rows, X, x_dtype == CRVQ_F32 ? ET_F32 : ET_F64, true, ld, X,
                                    x_dtype == CRVQ_F32 ? ET_F32 : ET_F64, ld, H, ldh, static_cast<hipStream_t>(stream)),
                    fn);
}

size_t crvq_hessian_inverse_workspace_size(int64_t N) {
  if (N < 1 || N > 65536) return 0;
  return hinv_ws_bytes(N);
}

crvq_status crvq_hessian_inverse_diagonal(const double* H, int64_t ldh, int64_t N, double damp, double* hinv,
                                          float* scale, void* workspace, size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_hessian_inverse_diagonal");
  static const char* fn = "crvq_hessian_inverse_diagonal";
  g_err.clear();
  if (N < 0 || N > 65536) return fail(CRVQ_ERR_INVALID, "%s: N = %lld outside [0, 65536]", fn, (long long)N);
  if (ldh < N) return fail(CRVQ_ERR_INVALID, "%s: ldh must be >= N", fn);
  if (!(damp >= 0.0 && damp < INFINITY)) return fail(CRVQ_ERR_INVALID, "%s: damp must be finite and >= 0", fn);
  if (N == 0) return CRVQ_OK;
  if (!H || (!hinv && !scale)) return fail(CRVQ_ERR_INVALID, "%s: H and one of hinv, scale must not be NULL", fn);
  crvq_status s = check_ws(workspace, ws_bytes, crvq_hessian_inverse_workspace_size(N), fn);
  if (s) return s;
  return hip_status(launch_hinv(H, ldh, N, damp, hinv, scale, workspace, static_cast<hipStream_t>(stream)), fn);
}

crvq_status crvq_hessian_product(int64_t M, int64_t N, int64_t n_out, const double* R, int64_t ldr, const double* H,
                                 int64_t ldh, double* G, int64_t ldg, double* row_loss, double* loss_total,
                                 void* stream) {
  const ApiRange range("crvq_hessian_product");
  static const char* fn = "crvq_hessian_product";
  g_err.clear();
  if (M < 0 || N < 1 || n_out < 1 || n_out > N) return fail(CRVQ_ERR_INVALID, "%s: need M >= 0 and 1 <= n_out <= N", fn);
  if (ldr < N || ldh < N || ldg < n_out) return fail(CRVQ_ERR_INVALID, "%s: ldr, ldh >= N and ldg >= n_out needed", fn);
  if (row_loss && n_out != N) return fail(CRVQ_ERR_INVALID, "%s: row_loss needs n_out == N", fn);
  if (loss_total && !row_loss) return fail(CRVQ_ERR_INVALID, "%s: loss_total needs row_loss", fn);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (M == 0) return loss_total ? hip_status(launch_sum_f64(0, nullptr, loss_total, st), fn) : CRVQ_OK;
  if (!R || !H || !G) return fail(CRVQ_ERR_INVALID, "%s: R, H and G must not be NULL", fn);
  crvq_status s = hip_status(launch_gemm_f64(M, n_out, N, R, ET_F64, false, ldr, H, ET_F64, ldh, G, ldg, st), fn);
  if (s || !row_loss) return s;
  if ((s = hip_status(launch_row_dot(M, N, R, ldr, G, ldg, row_loss, st), fn)) || !loss_total) return s;
  return hip_status(launch_sum_f64(M, row_loss, loss_total, st), fn);
}

size_t crvq_code_sums_workspace_size(int64_t n_vectors, int32_t d, int64_t K) {
  if (n_vectors < 0 || d < 1 || d > CRVQ_MAX_D || K < 1 || K > CRVQ_MAX_K) return 0;
  return code_sums_ws_bytes(n_vectors, K, d);
}

crvq_status crvq_code_sums(const double* X, int64_t n_rows, int64_t vecs_per_row, int64_t ld, int32_t d,
                           const int32_t* codes, int64_t K, double* sums, int32_t* counts, void* workspace,
                           size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_code_sums");
  static const char* fn = "crvq_code_sums";
  g_err.clear();
  if (d < 1 || d > CRVQ_MAX_D) return fail(CRVQ_ERR_UNSUPPORTED, "%s: d = %d outside [1, %d]", fn, d, CRVQ_MAX_D);
  if (n_rows < 0 || vecs_per_row < 0) return fail(CRVQ_ERR_INVALID, "%s: negative n_rows or vecs_per_row", fn);
  if (ld < vecs_per_row * d) return fail(CRVQ_ERR_INVALID, "%s: ld < vecs_per_row * d", fn);
  if (K < 1 || K > CRVQ_MAX_K) return fail(CRVQ_ERR_UNSUPPORTED, "%s: K = %lld outside [1, %d]", fn, (long long)K, CRVQ_MAX_K);
  const int64_t n = n_rows * vecs_per_row;
  if (n > 0x7fffffffLL) return fail(CRVQ_ERR_UNSUPPORTED, "%s: too many vectors", fn);
  if (!sums || (n > 0 && (!X || !codes))) return fail(CRVQ_ERR_INVALID, "%s: X, codes and sums must not be NULL", fn);
  crvq_status s = check_ws(workspace, ws_bytes, code_sums_ws_bytes(n, K, d), fn);
  if (s) return s;
  return hip_status(launch_code_sums(X, vecs_per_row > 0 ? vecs_per_row : 1, ld, d, n, codes, K, sums, counts,
                                     workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

crvq_status crvq_adam_step(float* C, const double* grad, double grad_scale, double* m, double* v, int64_t n,
                           int64_t step, double lr, double beta1, double beta2, double eps, void* stream) {
  const ApiRange range("crvq_adam_step");
  static const char* fn = "crvq_adam_step";
  g_err.clear();
  if (n < 0 || step < 1) return fail(CRVQ_ERR_INVALID, "%s: need n >= 0 and step >= 1", fn);
  if (!(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) || !(eps >= 0.0))
    return fail(CRVQ_ERR_INVALID, "%s: need 0 <= beta1, beta2 < 1 and eps >= 0", fn);
  if (n == 0) return CRVQ_OK;
  if (!C || !grad || !m || !v) return fail(CRVQ_ERR_INVALID, "%s: C, grad, m and v must not be NULL", fn);
  const double bc1 = 1.0 - std::pow(beta1, static_cast<double>(step));
  const double bc2 = 1.0 - std::pow(beta2, static_cast<double>(step));
  return hip_status(launch_adam(n, C, grad, grad_scale, m, v, lr, beta1, beta2, bc1, bc2, eps,
                                static_cast<hipStream_t>(stream)),
                    fn);
}

crvq_status crvq_adam_step_bf16(uint16_t* C, float* master, const double* grad, double grad_scale, double* m,
                                double* v, int64_t n, int64_t step, double lr, double beta1, double beta2, double eps,
                                void* stream) {
  const ApiRange range("crvq_adam_step_bf16");
  static const char* fn = "crvq_adam_step_bf16";
  g_err.clear();
  if (n < 0 || step < 1) return fail(CRVQ_ERR_INVALID, "%s: need n >= 0 and step >= 1", fn);
  if (!(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) || !(eps >= 0.0))
    return fail(CRVQ_ERR_INVALID, "%s: need 0 <= beta1, beta2 < 1 and eps >= 0", fn);
  if (n == 0) return CRVQ_OK;
  if (!C || !master || !grad || !m || !v)
    return fail(CRVQ_ERR_INVALID, "%s: C, master, grad, m and v must not be NULL", fn);
  const double bc1 = 1.0 - std::pow(beta1, static_cast<double>(step));
  const double bc2 = 1.0 - std::pow(beta2, static_cast<double>(step));
  return hip_status(launch_adam_bf16(n, C, master, grad, grad_scale, m, v, lr, beta1, beta2, bc1, bc2, eps, step == 1,
                                     static_cast<hipStream_t>(stream)),
                    fn);
}

size_t crvq_refine_workspace_size(int64_t M, int64_t N, int64_t n_cols) {
  if (M < 1 || n_cols < 1 || N < n_cols) return 0;
  return refine_ws_bytes(M, n_cols, N);
}

crvq_status crvq_refine_codes(int64_t M, int64_t N, int32_t d, int64_t n_cols, double* R, int64_t ldr, const double* H,
                              int64_t ldh, const void* C, int c_dtype, int64_t K, int32_t* codes, int64_t ldq,
                              void* workspace, size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_refine_codes");
  static const char* fn = "crvq_refine_codes";
  g_err.clear();
  if (M < 0 || N < 1) return fail(CRVQ_ERR_INVALID, "%s: need M >= 0 and N >= 1", fn);
  if (d < 1 || d > CRVQ_MAX_D) return fail(CRVQ_ERR_UNSUPPORTED, "%s: d = %d outside [1, %d]", fn, d, CRVQ_MAX_D);
  if (n_cols < 0 || n_cols > N || n_cols % d || N % d)
    return fail(CRVQ_ERR_INVALID, "%s: n_cols must be a multiple of d in [0, N] and d must divide N", fn);
  if (!dtype_ok(c_dtype)) return fail(CRVQ_ERR_INVALID, "%s: c_dtype must be F32 or BF16", fn);
  if (K < 1 || K > CRVQ_MAX_K) return fail(CRVQ_ERR_UNSUPPORTED, "%s: K = %lld outside [1, %d]", fn, (long long)K, CRVQ_MAX_K);
  if (ldr < N || ldh < N || ldq < n_cols / d) return fail(CRVQ_ERR_INVALID, "%s: ldr, ldh >= N and ldq >= n_cols / d", fn);
  if (M == 0 || n_cols == 0) return CRVQ_OK;
  if (!R || !H || !C || !codes) return fail(CRVQ_ERR_INVALID, "%s: R, H, C and codes must not be NULL", fn);
  crvq_status s = check_ws(workspace, ws_bytes, crvq_refine_workspace_size(M, N, n_cols), fn);
  if (s) return s;
  return hip_status(launch_refine_book(M, N, d, n_cols, R, ldr, H, ldh, C, c_dtype, K, codes, ldq, workspace,
                                       static_cast<hipStream_t>(stream)),
                    fn);
}

}  // extern "C"

// ------------------------------------------------------------------------------------------------
size_t crvq_gemv_workspace_size(int64_t M, int64_t N, int64_t K_base) {
  if (M < 1 || N < 64 || K_base < 1 || K_base > 256) return 0;
  return gemv_ws_bytes(M, N, static_cast<int>(K_base));
}

size_t crvq_workspace_size(int op, int64_t n_vectors, int64_t K, int32_t beam, int32_t n_books, int32_t d,
                           const int64_t* Ks, int64_t M, int64_t N, int64_t n_cols) {
  switch (op) {
    case CRVQ_OP_IMPORTANCE: return crvq_importance_workspace_size(M, N);
    case CRVQ_OP_REORDER: return crvq_reorder_workspace_size(N);
    case CRVQ_OP_ASSIGN: return crvq_assign_workspace_size(n_vectors, d, K);
    case CRVQ_OP_BEAM: return crvq_beam_workspace_size(n_vectors, d, n_books, Ks, beam);
    case CRVQ_OP_KMEANS: return crvq_kmeans_workspace_size(n_vectors, d, K);
    case CRVQ_OP_DEQUANT: return crvq_dequant_workspace_size(N);
    case CRVQ_OP_CODE_SUMS: return crvq_code_sums_workspace_size(n_vectors, d, K);
    case CRVQ_OP_REFINE: return crvq_refine_workspace_size(M, N, n_cols);
    case CRVQ_OP_GEMV: return crvq_gemv_workspace_size(M, N, K);
    case CRVQ_OP_HINV: return crvq_hessian_inverse_workspace_size(N);
    default: return 0;
  }
}

crvq_status crvq_dequant_gemv(int64_t M, int64_t N, int64_t n_crit, const uint8_t* q_base, int64_t ldq_base,
                              const void* C_base, int base_dtype, int64_t K_base, int32_t n_ext,
                              const uint8_t* const* q_ext, int64_t ldq_ext, const void* const* C_ext,
                              const int32_t* ext_dtypes, const int64_t* K_ext, const int32_t* perm, const void* x,
                              int x_dtype, float* y, void* workspace, size_t ws_bytes, void* stream) {
  const ApiRange range("crvq_dequant_gemv");
  static const char* fn = "crvq_dequant_gemv";
  g_err.clear();
  if (M < 0 || N < 1) return fail(CRVQ_ERR_INVALID, "%s: need M >= 0 and N >= 1", fn);
  if (N % 64) return fail(CRVQ_ERR_UNSUPPORTED, "%s: N = %lld is not a multiple of 64", fn, (long long)N);
  if (n_crit < 0 || n_crit > N || n_crit % 8)
    return fail(CRVQ_ERR_INVALID, "%s: n_crit = %lld must be a multiple of 8 in [0, N]", fn, (long long)n_crit);
  if (M == 0) return CRVQ_OK;  // no rows: nothing to compute or write
  if (!q_base || !C_base || !x || !y) return fail(CRVQ_ERR_INVALID, "%s: q_base, C_base, x and y must not be NULL", fn);
  if (!dtype_ok(base_dtype) || !dtype_ok(x_dtype)) return fail(CRVQ_ERR_INVALID, "%s: invalid base or x dtype", fn);
  if (K_base < 1 || K_base > 256) return fail(CRVQ_ERR_UNSUPPORTED, "%s: K_base = %lld outside [1, 256] (8-bit codes)", fn, (long long)K_base);
  if (ldq_base < N / 8 || ldq_base % 8 || (reinterpret_cast<uintptr_t>(q_base) & 7))
    return fail(CRVQ_ERR_INVALID, "%s: q_base must be 8-byte aligned with ldq_base >= N/8 and a multiple of 8", fn);
  if (n_ext < 0 || n_ext > CRVQ_MAX_BOOKS - 1)
    return fail(CRVQ_ERR_INVALID, "%s: n_ext = %d outside [0, %d]", fn, n_ext, CRVQ_MAX_BOOKS - 1);
  GemvExt ext = {};
  ext.n = n_ext;
  ext.ldq = ldq_ext;
  if (n_ext > 0) {
    if (!q_ext || !C_ext || !ext_dtypes || !K_ext)
      return fail(CRVQ_ERR_INVALID, "%s: q_ext, C_ext, ext_dtypes and K_ext must not be NULL when n_ext > 0", fn);
    if (ldq_ext < n_crit / 8) return fail(CRVQ_ERR_INVALID, "%s: ldq_ext < n_crit / 8", fn);
    for (int e = 0; e < n_ext; ++e) {
      if (!q_ext[e] || !C_ext[e]) return fail(CRVQ_ERR_INVALID, "%s: q_ext[%d] or C_ext[%d] is NULL", fn, e, e);
      if (!dtype_ok(ext_dtypes[e])) return fail(CRVQ_ERR_INVALID, "%s: ext_dtypes[%d] invalid", fn, e);
      if (K_ext[e] < 1 || K_ext[e] > 256)
        return fail(CRVQ_ERR_UNSUPPORTED, "%s: K_ext[%d] = %lld outside [1, 256] (8-bit codes)", fn, e, (long long)K_ext[e]);
      ext.C[e] = C_ext[e];
      ext.q[e] = q_ext[e];
      ext.type[e] = ext_dtypes[e];
      ext.K[e] = static_cast<int>(K_ext[e]);
    }
  }
  crvq_status s;
  if ((s = check_ws(workspace, ws_bytes, crvq_gemv_workspace_size(M, N, K_base), fn))) return s;
  return hip_status(launch_gemv(M, N, n_crit, q_base, ldq_base, C_base, base_dtype, static_cast<int>(K_base), ext, perm,
                                x, x_dtype, y, workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

crvq_status crvq_pack_codes_u8(const int32_t* codes, int64_t n, uint8_t* out, void* stream) {
  const ApiRange range("crvq_pack_codes_u8");
  static const char* fn = "crvq_pack_codes_u8";
  g_err.clear();
  if (n < 0) return fail(CRVQ_ERR_INVALID, "%s: n < 0", fn);
  if (n == 0) return CRVQ_OK;
  if (!codes || !out) return fail(CRVQ_ERR_INVALID, "%s: codes and out must not be NULL", fn);
  return hip_status(launch_pack_codes_u8(codes, n, out, static_cast<hipStream_t>(stream)), fn);
}
