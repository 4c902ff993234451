// Internal helpers shared by the kernels and the C-ABI layer of libkronq (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "kronq.h"

namespace kq {

// ---- error state (thread-local message behind kronq_last_error) ----------------------------
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

#define KQ_REQUIRE(cond, code, ...)      \
  do {                                   \
    if (!(cond)) {                       \
      ::kq::set_error(__VA_ARGS__);      \
      return (code);                     \
    }                                    \
  } while (0)

#define KQ_HIP(call)                                                              \
  do {                                                                            \
    hipError_t kq_e_ = (call);                                                    \
    if (kq_e_ != hipSuccess) {                                                    \
      ::kq::set_error("%s failed: %s", #call, hipGetErrorString(kq_e_));          \
      return KRONQ_ERR_HIP;                                                       \
    }                                                                             \
  } while (0)

#define KQ_TRY(expr)            \
  do {                          \
    int kq_rc_ = (expr);        \
    if (kq_rc_ != KRONQ_OK) {   \
      return kq_rc_;            \
    }                           \
  } while (0)

// ---- profiler: optional hipEvent pair around every launch ----------------------------------
bool prof_on();
bool prof_wants(const char* name);
void prof_begin(const char* name, hipStream_t s);
void prof_end(const char* name, hipStream_t s);

// Launch a kernel; checks the launch status and records profiler events when enabled.
template <typename Kernel, typename... Args>
int launch(const char* name, Kernel kernel, dim3 grid, dim3 block, size_t shmem, hipStream_t s,
           Args... args) {
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return KRONQ_OK;
  if (shmem > 65536) {  // opt in to more than 64 KB of dynamic LDS (gfx950 has 160 KB per CU)
    hipError_t ea = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                        hipFuncAttributeMaxDynamicSharedMemorySize, int(shmem));
    if (ea != hipSuccess) {
      set_error("LDS request of %zu bytes for %s refused: %s", shmem, name, hipGetErrorString(ea));
      return KRONQ_ERR_HIP;
    }
  }
  const bool p = prof_on() && prof_wants(name);
  if (p) prof_begin(name, s);
  hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("launch of %s failed: %s", name, hipGetErrorString(e));
    return KRONQ_ERR_HIP;
  }
  if (p) prof_end(name, s);
  return KRONQ_OK;
}

// ---- workspace carving -----------------------------------------------------------------------
struct Carver {
  char* base;
  size_t used = 0;
  explicit Carver(void* p) : base(static_cast<char*>(p)) {}
  template <typename T>
  T* take(size_t count) {
    used = (used + 255) & ~size_t(255);
    T* r = reinterpret_cast<T*>(base ? base + used : nullptr);
    used += count * sizeof(T);
    return r;
  }
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// compute units of the current device (cached per device; workgroup rounds are counted in them)
inline int device_cus() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cache[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        v <= 0)
      v = 256;
    cache[dev] = v;
  }
  return cache[dev];
}
inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---- shapes used by the rotation ---------------------------------------------------------------
// d = 2^k (k >= 1) -> (pow2 = d, has28 = false); d = 28 * 2^k -> (pow2 = 2^k, has28 = true).
struct RotDim {
  bool ok = false;
  bool has28 = false;
  int64_t m = 0;  // Hadamard order
};
RotDim rot_dim(int64_t d);

// ---- kernel-side entry points (defined in the per-step sources) ------------------------------
// covariance
// covariance (B == nullptr: H = A^T A, symmetric) or cross product (H = A^T B, all tiles)
size_t cov_ws_bytes(int dtype, int64_t n_rows, int64_t d, bool cross = false);
// max_cus > 0 caps the CUs the interior-tile launch holds at once (0: the whole chip)
int cov_launch(const void* A, const void* B, int dtype, int64_t n_rows, int64_t d, int64_t lda,
               float* H, int64_t ldh, float alpha, float beta, void* ws, hipStream_t s,
               int max_cus = 0);
// diag(A^T A) as column sums of squares (fp64 sums, one rounding to fp32)
size_t cov_diag_ws_bytes(int64_t n_rows, int64_t d);
// bytes of chunk partials a cov_diag launch with these sizes uses, and the address of this
// stream's device copy of the fixed scratch array of the no-allocation variant
size_t cov_diag_need_bytes(int64_t n_rows, int64_t d, int max_cus);
int cov_diag_scratch(hipStream_t s, void** out);
// register-resident bf16 MFMA loop (measured ceiling); *workgroups receives the grid size
int mfma_peak_launch(const uint16_t* data, int iters, float* out, int* workgroups, hipStream_t s);
int cov_diag_launch(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                    float* hdiag, int max_cus, void* ws, hipStream_t s);
// traces
int traces_launch(const float* HX, int64_t d_in, int64_t ldx, const float* HG, int64_t d_out,
                  int64_t ldg, double* out3, hipStream_t s);
// rotation
size_t rotate_ws_bytes(int64_t d_out, int64_t d_in);
int rotate_launch(const void* W_in, int w_dtype, int64_t ldw_in, float* W, int64_t d_out,
                  int64_t d_in, int64_t ldw, float* HX, int64_t ldx, float* HG, int64_t ldg,
                  const int8_t* sign_in, const int8_t* sign_out, const float* q28_in,
                  const float* q28_out, float* sx, float* sg, int flags, void* ws,
                  hipStream_t s);
// drift statistic: D <- V S_X^-1 D S_X^-1 V^T with the given sx
size_t rotate_drift_ws_bytes(int64_t d);
int rotate_drift_launch(float* D, int64_t d, int64_t ldd, const float* sx, const int8_t* sign,
                        const float* q28, int flags, void* ws, hipStream_t s);
// B vectors (rows of src) -> diag(post_col) T diag(pre_col) x, T the randomised Hadamard factor of
// order n (transposed with q_trans) when transform, else the identity
int rotate_vectors(const void* src, int dtype, int64_t lds, float* dst, int64_t ldd, int64_t rows,
                   int64_t n, const float* pre_col, const float* post_col, bool transform,
                   const float* q28, bool q_trans, hipStream_t s);
// mul = sign / s (sign NULL: 1; s NULL: 1)
int inverse_multipliers(const float* sv, const int8_t* sign, int64_t n, float* mul, hipStream_t s);
// online inference: packed codes and the packed-code GEMV
int pack_codes_launch(const uint8_t* codes, int64_t d_out, int64_t d_in, int64_t ldq, int bits,
                      uint32_t* packed, int64_t ldp, hipStream_t s);
size_t online_ws_bytes(int64_t d_out, int64_t d_in, int64_t batch);
int online_matvec_launch(const uint32_t* packed, int64_t ldp, const float* scales,
                         const float* zeros, int64_t ldsz, int bits, int group, int64_t d_out,
                         int64_t d_in, const float* mul_in, const float* mul_out,
                         const float* q28_in, const float* q28_out, int flags, const void* x,
                         int x_dtype, int64_t ldx, int64_t batch, float* y, int64_t ldy, void* ws,
                         hipStream_t s);
// diagnostics: matrix statistics, Jacobi eigendecomposition, expected-loss factors
size_t matrix_stats_ws_bytes(int64_t rows, int64_t cols);
int matrix_stats_launch(const void* M, int dtype, int64_t rows, int64_t cols, int64_t ld,
                        double* out, void* ws, hipStream_t s);
size_t eigh_ws_bytes(int64_t d);
int eigh_launch(const float* H, int64_t d, int64_t ldh, int sweeps, float* evals, float* Q,
                int64_t ldq, double* off, void* ws, hipStream_t s);
size_t proxy_ws_bytes(int64_t d_out, int64_t d_in);
int proxy_launch(const float* HG, int64_t ldg, const void* W, int w_dtype, int64_t ldw,
                 int64_t d_out, int64_t d_in, const float* Hd, int64_t ldh, const float* U,
                 int64_t ldu, const double* alphas, int n_alpha, double* out, void* ws,
                 hipStream_t s);
// fp32 GEMM on MFMA: C = alpha * op(A) op(B) + beta * C
enum GemmFlags : int {
  GEMM_TA = 1,          // op(A) = A^T (A stored [K x M])
  GEMM_TB = 2,          // op(B) = B^T (B stored [N x K])
  GEMM_LOWER_C = 4,     // only output tiles that touch the lower triangle (i >= j)
  GEMM_B_LOWER = 8,     // B is lower triangular: skip k < column-tile start
  GEMM_A_LOWER = 16,    // A is lower triangular: skip k > row-tile end
  GEMM_OPB_UPPER = 32,  // op(B) is upper triangular: skip k > column-tile end
  GEMM_UPPER_C = 64,    // only output tiles that touch the upper triangle (i <= j)
  GEMM_A_UPPER = 128,   // A is upper triangular: skip k < row-tile start
};
// C -= A B (+ A2 B2), A fp32 [M x K] (k contiguous), B given as the bf16 three-term split of
// B^T (Bh + Bl, [N x K], k contiguous); likewise A2 [M x K2], B2; K % 32 == 0, K2 % 32 == 0
struct Bf16x3Pair {
  const float* A = nullptr;
  int64_t lda = 0;
  const uint16_t* Bh = nullptr;
  const uint16_t* Bl = nullptr;
  int64_t ldb = 0;
  int64_t K = 0;
};
int gemm_bf16x3_sub(int64_t M, int64_t N, const Bf16x3Pair& p1, const Bf16x3Pair& p2, float* C,
                    int64_t ldc, hipStream_t s, const char* name);
// C -= (Ah + Al)(Bh + Bl)^T (three bf16 products) for operands split beforehand, [row][k]
int gemm_bf16x3_presplit_sub(int64_t M, int64_t N, int64_t K, const uint16_t* Ah,
                             const uint16_t* Al, int64_t lda, const uint16_t* Bh,
                             const uint16_t* Bl, int64_t ldb, float* C, int64_t ldc,
                             hipStream_t s, const char* name);
// Th + Tl = sign * U^T split into bf16 high and low parts, [d x d] with row stride ldt
// (sign = -1 when neg)
int split_transpose_launch(const float* U, int64_t ldu, int64_t d, uint16_t* Th, uint16_t* Tl,
                           int64_t ldt, hipStream_t s, bool neg = false, uint16_t* Fh = nullptr,
                           uint16_t* Fl = nullptr);

// Position of element (r, k) of a bf16 matrix kept in MFMA-fragment order for the operands of
// v_mfma_f32_32x32x16_bf16: 32 rows x 16 k form one 1 KB unit in which lane
// (r % 32) + 32 ((k % 16) / 8) holds its 8 consecutive k, so that a wave's fragment load is
// one contiguous kilobyte; the units of a 32-row group follow each other along k (ksteps units
// per group).
__host__ __device__ inline int64_t split_frag_index(int64_t r, int64_t k, int64_t ksteps) {
  return (((r >> 5) * ksteps + (k >> 4)) * 64 + (r & 31) + 32 * ((k >> 3) & 1)) * 8 + (k & 7);
}
// fp32-accurate C = alpha op(A) op(B) + beta C on the bf16 matrix cores (six-term split; the
// large products of the factorisation). Supported: not GEMM_TA, GEMM_UPPER_C or GEMM_A_UPPER;
// K, lda, ldb (and N when B is stored [K][N]) multiples of 4; A and B 16-byte aligned.
bool gemm_split6_supports(int flags, int64_t M, int64_t N, int64_t K, const float* A,
                          int64_t lda, const float* B, int64_t ldb);
int gemm_f32(int flags, int64_t M, int64_t N, int64_t K, float alpha, const float* A,
             int64_t lda, const float* B, int64_t ldb, float beta, float* C, int64_t ldc,
             hipStream_t s, const char* name = "gemm_f32_mfma");
// one product C = alpha op(A) op(B) + beta C with the GEMM_* flags
struct GemmProb {
  int flags;
  int64_t M, N, K;
  float alpha;
  const float* A;
  int64_t lda;
  const float* B;
  int64_t ldb;
  float beta;
  float* C;
  int64_t ldc;
};
// two independent products in one launch (small-tile kernel; the outputs must not overlap
// each other or the inputs)
int gemm_f32_dual(const GemmProb& p1, const GemmProb& p2, hipStream_t s, const char* name);
int gemm_f32_split6(int flags, int64_t M, int64_t N, int64_t K, float alpha, const float* A,
                    int64_t lda, const float* B, int64_t ldb, float beta, float* C, int64_t ldc,
                    hipStream_t s, const char* name);
// two independent products of the split path in one launch (the outputs must not overlap);
// the first product's workgroups are dispatched first
int gemm_f32_split6_dual(const GemmProb& p0, const GemmProb& p1, hipStream_t s,
                         const char* name);
// Cholesky inverse factor
size_t chol_ws_bytes(int64_t d);
int chol_launch(float* H, int64_t d, int64_t ldh, float damp_rel, float* U, int64_t ldu,
                int* info, void* ws, hipStream_t s);
// drift correction P = alpha ((D U^T) . M_U) U
size_t gptaq_ws_bytes(int64_t d);
int gptaq_launch(const float* D, int64_t d, int64_t ldd, const float* U, int64_t ldu, float alpha,
                 float* P, int64_t ldp, void* ws, hipStream_t s);
// OBS sweep (P == nullptr: no drift correction)
size_t obs_ws_bytes(int64_t d_out, int64_t d_in, bool drift);
int obs_group_ok(int64_t d_in, int group);
int obs_launch(float* W, int64_t d_out, int64_t d_in, int64_t ldw, const float* U, int64_t ldu,
               int bits, int group, const float* P, int64_t ldp, uint8_t* codes, float* scales,
               float* zeros, float* err, float* W_hat, void* ws, hipStream_t s);
// loss
size_t loss_ws_bytes(int64_t d_out, int64_t d_in);
int loss_launch(const void* W, int w_dtype, int64_t ldw, const float* W_hat, int64_t ldwh,
                int64_t d_out, int64_t d_in, const float* HX, int64_t ldx, const float* HG,
                int64_t ldg, double* loss, void* ws, hipStream_t s);

}  // namespace kq
