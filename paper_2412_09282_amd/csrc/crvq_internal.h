// Internal declarations shared by the host API and the kernel translation units of libcrvq.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace crvq {

enum ElemType : int { ET_F32 = 0, ET_BF16 = 1, ET_F64 = 2 };

constexpr int kMaxBeam = 16;
constexpr int kMaxBooks = 8;

// Output code arrays of the beam search, one per codebook.
struct CodePtrs {
  int32_t* q[kMaxBooks];
  int64_t ld[kMaxBooks];
};

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Streaming loads and stores of data touched once (whole weight matrices, code arrays, outputs).
// The nontemporal hint keeps such streams from displacing reused data in L2 and the last-level
// cache and lets the memory system stream them: a plain read of a 940 MB array runs at about
// 4 TB/s on MI355X, the same read with nontemporal loads at about 5.4 TB/s.
#ifndef CRVQ_NT_STORE
#define CRVQ_NT_STORE 1
#endif
typedef unsigned int crvq_u4 __attribute__((ext_vector_type(4)));
typedef unsigned int crvq_u2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint4 ld_stream(const void* p) {
  const crvq_u4 t = __builtin_nontemporal_load(static_cast<const crvq_u4*>(p));
  return make_uint4(t[0], t[1], t[2], t[3]);
}
__device__ __forceinline__ uint2 ld_stream8(const void* p) {
  const crvq_u2 t = __builtin_nontemporal_load(static_cast<const crvq_u2*>(p));
  return make_uint2(t[0], t[1]);
}
__device__ __forceinline__ int ld_stream_i32(const int* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_stream(void* p, uint4 v) {
  if (CRVQ_NT_STORE) {
    const crvq_u4 t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, static_cast<crvq_u4*>(p));
  } else {
    *static_cast<uint4*>(p) = v;
  }
}
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Bump allocator over a caller-supplied workspace (or a dry run that only measures).
struct WsCursor {
  char* base;
  size_t used = 0;
  explicit WsCursor(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(size_t count) {
    size_t off = used;
    used = align256(used + count * sizeof(T));
    return base ? reinterpret_cast<T*>(base + off) : nullptr;
  }
};

// A set of rows of length d read by the distance kernels.  Either a vector set over a matrix
// (ET_F32 / ET_BF16: row v = r * vpr + g at element r * ld + g * d) or a dense fp64 array of
// rows (ET_F64: row v at element v * d).
struct RowSrc {
  const void* base;
  int type;
  int d;
  int64_t vpr;
  int64_t ld;
  int64_t n;
};

// ---- codebook screen (k_screen.hip) -------------------------------------------------------------
struct ScreenPlan {
  int nb;            // best tiles tracked per lane (power of two >= requested top count)
  int cb;            // 16-row column blocks per wave
  int ks;            // 4-wide K steps of the fp32 MFMA (ceil(d / 4)); 2 (8 dimensions) when split
  int split;         // 1: split-bf16 MFMA screen (d <= 8), 0: fp32 MFMA screen
  int chunk;         // top-1: tiles per tracking chunk (1 = single tiles)
  int s32;           // 1: top-1 screen on 32 x 32 split-fp16 tiles (tiles then count 32 codewords)
  int prune;         // 1 (s32 only): codebook and rows in key order, certified chunk skipping
  int64_t tiles;     // 16-codeword tiles (ceil(K / 16))
  int64_t grid_x;    // row groups
  int splits;        // codebook splits (grid y)
  int64_t tiles_per_split;
};
ScreenPlan plan_screen(int64_t n_rows, int d, int64_t K, int top);

struct ScreenWs {
  float* apack;  // codebook in MFMA A-operand order, tiles x 64 lanes x ks
  float* cnp;    // ||c||^2 per codeword, +inf for padding
  int* pT;       // top-B: kept tile ids, [split][lane group][nb][row]
  float* pM;     // top-B: their screen minima, same layout
  float* pR;     // smallest screen value outside the exactly scored codewords, [split][row]
  double* pD;    // top-1: exact distance of the split's winner, [split][row]
  int* pK;       // top-1: its codeword, [split][row]
  double* xn2;   // top-1: ||x||^2 per row (fp64)
  float* xe;     // 32 x 32 top-1 screen on fp16-rounded operands: per row the factor of R in its bound's
                 // split term (written by the first screen)
  float* smax;   // 32 x 32 screen: partial maxima of |c|, then the scale alpha
  int* rcount;   // number of rows that failed the certification ([1]: that failed the second screen)
  int* rlist;    // those rows (any order), [n_rows]
  int* rlist2;   // 32 x 32 screen on inexact operands: rows that failed the second screen too, [n_rows
                 // rounded up to 256]; first the per-block slices of the first screen's failures
  int* bcount;   // their per-block counts, then the blocks' offsets, [2 x blocks of 256 rows]
  // pruned screen (prune): key order of codewords and rows, chunk ranges, binning parameters
  int* corder;   // sorted codeword position -> codeword [tiles x 32]
  int* ckey;     // codeword keys [K]
  int* coff;     // first sorted position of every key [16384]
  int* hist;     // key counts then cursors, codewords [16384] and rows [16384]; then the fine
                 // histograms of the three key features over the codebook [3 x 4096]
  uint4* cbnd;   // chunk ranges of the norm and coordinate j [tiles / 2]
  uint2* cbnd3;  // chunk ranges of coordinate q [tiles / 2]
  uint32_t* cminS;
  uint32_t* cmaxP;
  float* prm;    // binning parameters and the scaled largest codeword norm [6], then partial ranges
  int* rkey;     // row keys [n_rows]
  int* rord;     // rows in key order [n_rows]
  float* tD;     // the first screen's exact distance of each uncertain row, per-block slices [n_rows
                 // rounded up to 256], then compacted beside the row list into lD [n_rows]
  float* lD;
};
// Carves the screen's scratch out of `ws`; returns it (pointers null on a dry run).
ScreenWs carve_screen(WsCursor& ws, const ScreenPlan& p, int64_t n_rows, int64_t K_alloc);

// Prepares the codebook, runs the MFMA screen and the exact finalize (with rescue).  When
// out_codes != nullptr (top == 1) writes codes / dist; otherwise writes the sorted top-`top`
// (D, k) lists per row to rowD / rowK (row-major [n_rows][top]).
hipError_t launch_screen(const RowSrc& src, const void* C, int c_type, int64_t K, int top, const ScreenPlan& p,
                         const ScreenWs& w, int32_t* out_codes, float* out_dist, double* rowD, int* rowK,
                         hipStream_t stream);

// Beam bookkeeping kernels.
hipError_t launch_beam_merge(int64_t n, int n_par, int beam, int step, int n_books, const double* rowD,
                             const int* rowK, const RowSrc& src0, const double* res_in, double* res_out,
                             const int* tup_in, int* tup_out, double* err_out, const void* book, int book_type,
                             int64_t K, int d, hipStream_t stream);
hipError_t launch_beam_emit(int64_t n, int64_t vpr, int n_par, int n_books, const int* tup, const double* err,
                            const CodePtrs& outs, float* err_out, hipStream_t stream);

// ---- K-means update (k_kmeans.hip) -------------------------------------------------------------
size_t kmeans_ws_bytes(int64_t n, int64_t K);
hipError_t launch_kmeans_update(const RowSrc& src, const int32_t* codes, int64_t K, void* C, int c_type,
                                int32_t* counts, void* ws, hipStream_t stream);

// ---- column reduction (k_colreduce.hip) --------------------------------------------------------
size_t colreduce_ws_bytes(int64_t M, int64_t N);
hipError_t launch_colreduce(const void* A, int64_t lda, const void* B, int64_t ldb, int type, int64_t M, int64_t N,
                            const float* scale, int reduce, float* out, void* ws, hipStream_t stream);

// ---- reorder / gathers (k_reorder.hip) -----------------------------------------------------------
int rank_chunks(int64_t N);
// part: int32 scratch of rank_chunks(N) * N entries
hipError_t launch_rank_perm(const float* importance, int64_t N, int32_t* perm, int32_t* part, hipStream_t stream);
hipError_t launch_inverse_perm(const int32_t* perm, int64_t N, int32_t* inv, hipStream_t stream);
hipError_t launch_gather_columns(const void* in, int64_t ld_in, void* out, int64_t ld_out, int esize, int64_t M,
                                 int64_t N, const int32_t* src_idx, hipStream_t stream);
hipError_t launch_gather_vectors(const RowSrc& src, const int64_t* idx, int64_t count, void* out, int out_type,
                                 hipStream_t stream);

// ---- dequant (k_dequant.hip) ---------------------------------------------------------------------
struct DequantBooks {
  const void* C[8];
  const int32_t* q[8];
  int type[8];
  int64_t K[8];
  int n;             // books in use (1 = basic only)
  int n_full;        // leading books that cover every vector (the basic books); the rest cover critical groups
  int64_t ldq_base;  // row stride of the code arrays of the first n_full books
  int64_t ldq_ext;   // row stride of the code arrays of the others
};
hipError_t launch_dequant(int64_t M, int64_t n_cols, int d, int64_t n_crit, const DequantBooks& books,
                          const int32_t* inv_perm, const int32_t* perm, const void* minuend, int min_type,
                          int64_t ld_min, void* out, int out_type, int64_t ld_out, hipStream_t stream);

// ---- matrix-vector product with a quantized layer (k_gemv.hip) -----------------------------------
struct GemvExt {
  const void* C[8];
  const uint8_t* q[8];
  int type[8];
  int K[8];
  int n;        // extended books
  int64_t ldq;  // row stride of their code arrays
};
struct GemvPlan {
  int G;                   // groups per lane; a slice is 16 G groups
  int fused;               // 1: the finishing kernel looks the extended codes up in LDS tables
  int n_slices;
  size_t lds;              // bytes of LDS per slice workgroup (table, xs)
  size_t ext_lds;          // bytes of LDS of the extended-book workgroups' tables
  int ext_cols;            // columns of workgroups for the extended books (0: none)
  int64_t rows_per_block;  // a multiple of 32
  int64_t row_blocks;
};
GemvPlan plan_gemv(int64_t M, int64_t N, int K_base, int64_t ncv, int ext_K_sum, int n_ext);
size_t gemv_ws_bytes(int64_t M, int64_t N, int K_base);
hipError_t launch_gemv(int64_t M, int64_t N, int64_t n_crit, const uint8_t* q_base, int64_t ldq_base, const void* C_base,
                       int base_type, int K_base, const GemvExt& ext, const int32_t* perm, const void* x, int x_type,
                       float* y, void* ws, hipStream_t stream);
hipError_t launch_pack_codes_u8(const int32_t* codes, int64_t n, uint8_t* out, hipStream_t stream);

// ---- loss-driven refinement (k_refine.hip) ---------------------------------------------------------
hipError_t launch_gemm_f64(int64_t M, int64_t Nc, int64_t Kd, const void* A, int a_type, bool trans_a, int64_t lda,
                           const void* B, int b_type, int64_t ldb, double* C, int64_t ldc, hipStream_t stream,
                           bool sub = false);
hipError_t launch_row_dot(int64_t M, int64_t n, const double* A, int64_t lda, const double* B, int64_t ldb,
                          double* out, hipStream_t stream);
hipError_t launch_sum_f64(int64_t n, const double* x, double* out, hipStream_t stream);

// ---- inverse Hessian diagonal (k_hinv.hip) ------------------------------------------------------
size_t hinv_ws_bytes(int64_t N);
hipError_t launch_hinv(const double* H, int64_t ldh, int64_t N, double damp, double* hinv, float* scale, void* ws,
                       hipStream_t stream);
size_t code_sums_ws_bytes(int64_t n, int64_t K, int d);
size_t code_sums_large_ws_bytes(int64_t n, int64_t K);
hipError_t launch_code_sums_large(const RowSrc& src, const int32_t* codes, int64_t K, double* sums, int32_t* counts,
                                  void* ws, hipStream_t stream);
hipError_t launch_code_sums(const double* X, int64_t vpr, int64_t ld, int d, int64_t n, const int32_t* codes,
                            int64_t K, double* sums, int32_t* counts, void* ws, hipStream_t stream);
hipError_t launch_adam_bf16(int64_t n, uint16_t* C, float* master, const double* grad, double scale, double* m,
                            double* v, double lr, double b1, double b2, double bc1, double bc2, double eps, bool first,
                            hipStream_t stream);
hipError_t launch_adam(int64_t n, float* C, const double* grad, double scale, double* m, double* v, double lr,
                       double b1, double b2, double bc1, double bc2, double eps, hipStream_t stream);
size_t refine_lds_bytes(int64_t K, int d);
size_t refine_ws_bytes(int64_t M, int64_t n_cols, int64_t N);
hipError_t launch_refine_book(int64_t M, int64_t N, int d, int64_t n_cols, double* R, int64_t ldr, const double* H,
                              int64_t ldh, const void* Cb, int c_type, int64_t K, int32_t* codes, int64_t ldq,
                              void* ws, hipStream_t stream);

}  // namespace crvq
