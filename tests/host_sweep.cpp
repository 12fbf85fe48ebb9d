// Host-side sweep of libcrvq's planners and launch arithmetic over degenerate shapes, built with
// the library's sources compiled for the host only under -fsanitize=undefined (integer division by
// zero, overflow, bad shifts abort the run).  No GPU is used: device pointers are fake addresses that
// are never dereferenced on the host, and every launch fails for lack of a device, after the host has
// computed its grid, workspace layout and split plan.
//
// Covered: plan_screen / carve_screen for top 1..16, gemm_split_parts and the split-k GEMM launcher,
// the refinement, code-sum, K-means, column-reduction, reorder, dequant, GEMV and inverse-Hessian
// sizers, and every
// public entry point with shapes at and around the tile sizes (1, 15, 16, 17, 511, 512, 1024, ...),
// vector sets narrower than d, and n_cols below d.
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "crvq.h"
#include "crvq_internal.h"

namespace crvq {
int64_t gemm_split_parts(int64_t M, int64_t Nc, int64_t Kd);
hipError_t launch_gemm_f64_split(int64_t M, int64_t Nc, int64_t Kd, const double* A, int64_t lda, const double* B,
                                 int64_t ldb, double* C, int64_t ldc, double* ws, hipStream_t stream);
size_t kmeans_ws_bytes(int64_t n, int64_t K);
size_t colreduce_ws_bytes(int64_t M, int64_t N);
size_t gemv_ws_bytes(int64_t M, int64_t N, int K_base);
}  // namespace crvq

using namespace crvq;

// distinct 256-byte aligned addresses 2^40 apart, so no two fake arrays overlap
static void* fake(size_t i) { return reinterpret_cast<void*>((static_cast<uintptr_t>(i) + 1) << 40); }

static long long g_calls = 0, g_hip = 0;
static int g_bad = 0;

// A call on valid arguments may only succeed or fail in the runtime (no device here).
static void expect_ok_or_hip(int status, const char* what) {
  ++g_calls;
  if (status == CRVQ_ERR_HIP) ++g_hip;
  if (status != CRVQ_OK && status != CRVQ_ERR_HIP) {
    std::fprintf(stderr, "unexpected status %d from %s: %s\n", status, what, crvq_last_error());
    ++g_bad;
  }
}

int main() {
  const int64_t sizes[] = {1, 2, 7, 8, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129,
                           255, 256, 257, 511, 512, 513, 1023, 1024, 1025, 4096, 4097, 65536};
  const int64_t Ksizes[] = {1, 2, 15, 16, 17, 255, 256, 257, 4095, 4096, 4097, 8192, 65535, 65536};
  const int ds[] = {1, 3, 4, 5, 8, 9, 16};

  // planners
  for (int64_t n : sizes)
    for (int d : ds)
      for (int64_t K : Ksizes)
        for (int top : {1, 2, 3, 4, 8, 16}) {
          ScreenPlan p = plan_screen(n, d, K, top);
          WsCursor c(nullptr);
          carve_screen(c, p, n, K);
          if (p.splits < 1 || p.tiles_per_split < 1 || p.grid_x < 1) {
            std::fprintf(stderr, "plan_screen(%lld, %d, %lld, %d): splits %d tps %lld grid %lld\n", (long long)n, d,
                         (long long)K, top, p.splits, (long long)p.tiles_per_split, (long long)p.grid_x);
            ++g_bad;
          }
        }
  for (int64_t M : sizes)
    for (int64_t Nc : sizes)
      for (int64_t Kd : {int64_t{1}, int64_t{15}, int64_t{16}, int64_t{17}, int64_t{511}, int64_t{512},
                         int64_t{1024}, int64_t{1031}, int64_t{2049}, int64_t{4096}}) {
        const int64_t P = gemm_split_parts(M, Nc, Kd);
        if (P < 1) {
          std::fprintf(stderr, "gemm_split_parts(%lld, %lld, %lld) = %lld\n", (long long)M, (long long)Nc,
                       (long long)Kd, (long long)P);
          ++g_bad;
        }
        (void)launch_gemm_f64_split(M, Nc, Kd, static_cast<const double*>(fake(0)), Kd,
                                    static_cast<const double*>(fake(1)), Nc, static_cast<double*>(fake(2)), Nc,
                                    static_cast<double*>(fake(3)), nullptr);
        ++g_calls;
      }
  for (int64_t n : sizes)
    for (int64_t K : Ksizes) {
      (void)kmeans_ws_bytes(n, K);
      for (int d : ds) (void)crvq_code_sums_workspace_size(n, d, K);
    }
  for (int64_t M : sizes)
    for (int64_t N : sizes) {
      (void)colreduce_ws_bytes(M, N);
      (void)crvq_reorder_workspace_size(N);
      for (int64_t nc : {int64_t{1}, int64_t{8}, N}) (void)crvq_refine_workspace_size(M, N, nc);
      if (N % 64 == 0) (void)gemv_ws_bytes(M, N, 256);
      (void)crvq_hessian_inverse_workspace_size(N);
    }

  // every entry point on valid shapes (fake device pointers, enough workspace)
  void* X = fake(10);
  void* Cb = fake(11);
  int32_t* codes = static_cast<int32_t*>(fake(12));
  float* dist = static_cast<float*>(fake(13));
  void* ws = fake(14);
  const size_t big = size_t{1} << 40;
  for (int64_t rows : {int64_t{0}, int64_t{1}, int64_t{17}, int64_t{513}})
    for (int64_t vpr : {int64_t{1}, int64_t{3}, int64_t{16}})
      for (int d : ds)
        for (int64_t K : Ksizes) {
          expect_ok_or_hip(crvq_assign(X, CRVQ_F32, rows, vpr, vpr * d, d, Cb, CRVQ_F32, K, codes, dist, ws, big,
                                       nullptr),
                           "crvq_assign");
          expect_ok_or_hip(crvq_kmeans_update(X, CRVQ_BF16, rows, vpr, vpr * d + 1, d, codes, K, Cb, CRVQ_BF16,
                                              codes, ws, big, nullptr),
                           "crvq_kmeans_update");
          const int64_t Ks[3] = {K, 17, 256};
          const void* books[3] = {Cb, Cb, Cb};
          const int32_t dts[3] = {CRVQ_F32, CRVQ_F32, CRVQ_BF16};
          int32_t* cs[3] = {codes, codes, codes};
          for (int beam : {1, 2, 5, 16})
            expect_ok_or_hip(crvq_assign_residual_beam(X, CRVQ_F32, rows, vpr, vpr * d, d, 3, books, dts, Ks, beam,
                                                       cs, nullptr, dist, ws, big, nullptr),
                             "crvq_assign_residual_beam");
          expect_ok_or_hip(crvq_code_sums(static_cast<const double*>(X), rows, vpr, vpr * d, d, codes, K,
                                          static_cast<double*>(Cb), codes, ws, big, nullptr),
                           "crvq_code_sums");
        }
  for (int64_t M : {int64_t{1}, int64_t{15}, int64_t{16}, int64_t{17}, int64_t{511}, int64_t{512}, int64_t{1024}})
    for (int64_t N : {int64_t{8}, int64_t{16}, int64_t{64}, int64_t{128}, int64_t{1024}, int64_t{8200}}) {
      expect_ok_or_hip(crvq_channel_importance(X, N, nullptr, 0, CRVQ_F32, M, N, nullptr, CRVQ_REDUCE_SUM,
                                               dist, ws, big, nullptr),
                       "crvq_channel_importance");
      expect_ok_or_hip(crvq_reorder(X, N, fake(20), N, CRVQ_BF16, M, N, dist, codes, 1, ws, big, nullptr),
                       "crvq_reorder");
      for (int d : {1, 8, 16}) {
        if (N % d) continue;
        for (int64_t n_crit : {int64_t{0}, int64_t{d}, N}) {
          const int32_t* q[3] = {codes, codes, codes};
          const void* C[3] = {Cb, Cb, Cb};
          const int32_t dts[3] = {CRVQ_F32, CRVQ_F32, CRVQ_F32};
          const int64_t Ks[3] = {65536, 256, 256};
          for (int ne : {0, 1, 2})
            for (int use_perm : {0, 1}) {
              expect_ok_or_hip(crvq_dequant_books(M, N, d, n_crit, 1, ne, q, N / d, n_crit / d > 0 ? n_crit / d : 1,
                                                  C, dts, Ks, use_perm ? codes : nullptr, nullptr, 0, 0, fake(21),
                                                  CRVQ_F32, N, ws, big, nullptr),
                               "crvq_dequant_books");
            }
          for (int64_t Kr : {int64_t{d == 16 ? 512 : 256}, int64_t{4097}, int64_t{65536}})
            expect_ok_or_hip(crvq_refine_codes(M, N, d, n_crit, static_cast<double*>(fake(22)), N,
                                               static_cast<const double*>(fake(23)), N, Cb, CRVQ_F32, Kr, codes,
                                               N / d, ws, big, nullptr),
                             "crvq_refine_codes");
        }
      }
      expect_ok_or_hip(crvq_hessian_product(M, N, N, static_cast<const double*>(fake(22)), N,
                                            static_cast<const double*>(fake(23)), N, static_cast<double*>(fake(24)),
                                            N, static_cast<double*>(fake(25)), static_cast<double*>(fake(26)),
                                            nullptr),
                       "crvq_hessian_product");
      expect_ok_or_hip(crvq_gram(X, CRVQ_F32, M, N, N, static_cast<double*>(fake(24)), N, nullptr), "crvq_gram");
      expect_ok_or_hip(crvq_hessian_inverse_diagonal(static_cast<const double*>(fake(22)), N, N, 0.01,
                                                     static_cast<double*>(fake(28)), static_cast<float*>(fake(29)),
                                                     ws, big, nullptr),
                       "crvq_hessian_inverse_diagonal");
      if (N % 64 == 0)
        expect_ok_or_hip(crvq_dequant_gemv(M, N, 8, static_cast<const uint8_t*>(fake(27)), N / 8, Cb, CRVQ_BF16,
                                           256, 0, nullptr, 0, nullptr, nullptr, nullptr, codes, X, CRVQ_F32,
                                           dist, ws, big, nullptr),
                         "crvq_dequant_gemv");
    }
  if (g_bad) {
    std::fprintf(stderr, "host sweep: %d failures\n", g_bad);
    return 1;
  }
  std::printf("host sweep ok: %lld calls, %lld of them reached a launch\n", g_calls, g_hip);
  return 0;
}
