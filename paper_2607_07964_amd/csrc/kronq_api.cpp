// C-ABI entry points of libkronq: argument validation, workspace checks and dispatch to the
// HIP kernels. Nothing is enqueued when a check fails.
#include <hip/hip_runtime.h>

#include "kq_common.hpp"

namespace {

using kq::aligned;

bool valid_dtype(int t) { return t == KRONQ_BF16 || t == KRONQ_FP32; }

int check_ws(void* ws, size_t ws_bytes, size_t need) {
  KQ_REQUIRE(ws_bytes >= need, KRONQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given",
             need, ws_bytes);
  KQ_REQUIRE(need == 0 || (ws && aligned(ws, 256)), KRONQ_ERR_INVALID_ARG,
             "workspace must be a 256-byte aligned device pointer");
  return KRONQ_OK;
}

// fp32 matrix used with 16-byte vector accesses
int check_f32_mat(const float* p, int64_t rows, int64_t cols, int64_t ld, const char* what) {
  KQ_REQUIRE(p, KRONQ_ERR_INVALID_ARG, "%s is NULL", what);
  KQ_REQUIRE(rows >= 1 && cols >= 1, KRONQ_ERR_INVALID_ARG, "%s has a non-positive size", what);
  KQ_REQUIRE(ld >= cols, KRONQ_ERR_INVALID_ARG, "leading dimension of %s (%lld) < %lld", what,
             (long long)ld, (long long)cols);
  KQ_REQUIRE(ld % 4 == 0 && aligned(p, 16), KRONQ_ERR_INVALID_ARG,
             "%s must be 16-byte aligned with a leading dimension divisible by 4", what);
  return KRONQ_OK;
}

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

int check_cov_diag_args(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                        const float* hdiag, int max_cus) {
  KQ_REQUIRE(max_cus >= 0, KRONQ_ERR_INVALID_ARG, "max_cus must be >= 0");
  KQ_REQUIRE(valid_dtype(dtype), KRONQ_ERR_INVALID_ARG, "dtype must be KRONQ_BF16 or KRONQ_FP32");
  KQ_REQUIRE(hdiag && aligned(hdiag, 4), KRONQ_ERR_INVALID_ARG, "hdiag is NULL or misaligned");
  KQ_REQUIRE(n_rows >= 0 && d >= 1 && d <= (int64_t(1) << 24), KRONQ_ERR_INVALID_ARG,
             "need n_rows >= 0 and 1 <= d <= 2^24");
  if (n_rows > 0) {
    KQ_REQUIRE(A, KRONQ_ERR_INVALID_ARG, "A is NULL");
    KQ_REQUIRE(lda >= d, KRONQ_ERR_INVALID_ARG, "lda < d");
    KQ_REQUIRE(aligned(A, 16) && lda % (dtype == KRONQ_BF16 ? 8 : 4) == 0, KRONQ_ERR_INVALID_ARG,
               "A must be 16-byte aligned with lda divisible by 8 (bf16) or 4 (fp32)");
  }
  return KRONQ_OK;
}

constexpr int64_t kMaxRotDim = 32768;  // a transformed row must fit the 160 KB LDS

int check_rot_side(int64_t d, const int8_t* sign, const float* q28, const char* side) {
  const kq::RotDim r = kq::rot_dim(d);
  KQ_REQUIRE(r.ok && d <= kMaxRotDim, KRONQ_ERR_UNSUPPORTED,
             "%s dimension %lld is not 2^k or 28*2^k (<= %lld)", side, (long long)d,
             (long long)kMaxRotDim);
  KQ_REQUIRE(sign, KRONQ_ERR_INVALID_ARG, "%s rotation needs its sign vector", side);
  KQ_REQUIRE(!r.has28 || (q28 && aligned(q28, 4)), KRONQ_ERR_INVALID_ARG,
             "%s dimension %lld = 28 * 2^k needs the 28 x 28 factor", side, (long long)d);
  return KRONQ_OK;
}

}  // namespace

namespace {

int obs_common(float* W, int64_t d_out, int64_t d_in, int64_t ldw, const float* U, int64_t ldu,
               const float* P, int64_t ldp, int bits, int group, int block, uint8_t* codes,
               float* scales, float* zeros, float* err, float* W_hat, void* ws, size_t ws_bytes,
               void* stream) {
  KQ_REQUIRE(bits >= 2 && bits <= 8, KRONQ_ERR_UNSUPPORTED, "bits must be in 2..8");
  KQ_REQUIRE(block == 128, KRONQ_ERR_UNSUPPORTED, "only block size 128 is implemented");
  KQ_TRY(check_f32_mat(W, d_out, d_in, ldw, "W"));
  KQ_REQUIRE(group >= 1 && d_in % group == 0, KRONQ_ERR_SHAPE,
             "d_in (%lld) must be a multiple of the group (%d)", (long long)d_in, group);
  KQ_REQUIRE(kq::obs_group_ok(d_in, group) > 0, KRONQ_ERR_UNSUPPORTED,
             "group %d is not supported: it must be a multiple of 128 that divides d_in", group);
  KQ_TRY(check_f32_mat(U, d_in, d_in, ldu, "U"));
  if (P) KQ_TRY(check_f32_mat(P, d_in, d_in, ldp, "P"));
  KQ_REQUIRE(codes && aligned(codes, 4), KRONQ_ERR_INVALID_ARG, "codes must be 4-byte aligned");
  KQ_REQUIRE(scales && zeros && aligned(scales, 4) && aligned(zeros, 4), KRONQ_ERR_INVALID_ARG,
             "scales and zeros are required");
  KQ_REQUIRE(!err || aligned(err, 16), KRONQ_ERR_INVALID_ARG, "err must be 16-byte aligned");
  KQ_REQUIRE(!W_hat || aligned(W_hat, 16), KRONQ_ERR_INVALID_ARG,
             "W_hat must be 16-byte aligned");
  KQ_REQUIRE(static_cast<const float*>(W) != U && static_cast<const float*>(W) != P,
             KRONQ_ERR_INVALID_ARG, "W must not alias U or P");
  KQ_TRY(check_ws(ws, ws_bytes, kq::obs_ws_bytes(d_out, d_in, P != nullptr)));
  return kq::obs_launch(W, d_out, d_in, ldw, U, ldu, bits, group, P, ldp, codes, scales, zeros,
                        err, W_hat, ws, as_stream(stream));
}

}  // namespace

extern "C" {

size_t kronq_workspace_bytes(int op, int64_t d_out, int64_t d_in, int64_t n_rows) {
  switch (op) {
    case KRONQ_OP_COV:
      return kq::cov_ws_bytes(KRONQ_BF16, n_rows, d_in);
    case KRONQ_OP_CROSS:
      return kq::cov_ws_bytes(KRONQ_BF16, n_rows, d_in, true);
    case KRONQ_OP_COV_DIAG:
      return kq::cov_diag_ws_bytes(n_rows, d_in);
    case KRONQ_OP_ROTATE_DRIFT:
      return kq::rotate_drift_ws_bytes(d_in);
    case KRONQ_OP_GPTAQ:
      return kq::gptaq_ws_bytes(d_in);
    case KRONQ_OP_OBS_DRIFT:
      return kq::obs_ws_bytes(d_out, d_in, true);
    case KRONQ_OP_ONLINE:
      return kq::online_ws_bytes(d_out, d_in, n_rows);
    case KRONQ_OP_STATS:
      return kq::matrix_stats_ws_bytes(d_out, d_in);
    case KRONQ_OP_EIGH:
      return kq::eigh_ws_bytes(d_in);
    case KRONQ_OP_PROXY:
      return kq::proxy_ws_bytes(d_out, d_in);
    case KRONQ_OP_ROTATE:
      return kq::rotate_ws_bytes(d_out, d_in);
    case KRONQ_OP_CHOL:
      return kq::chol_ws_bytes(d_in);
    case KRONQ_OP_OBS:
      return kq::obs_ws_bytes(d_out, d_in, false);
    case KRONQ_OP_LOSS:
      return kq::loss_ws_bytes(d_out, d_in);
    default:
      return 0;
  }
}

int kronq_accumulate_cov(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                         float* H, int64_t ldh, float alpha, float beta, void* ws,
                         size_t ws_bytes, void* stream) {
  return kronq_accumulate_cov_limited(A, dtype, n_rows, d, lda, H, ldh, alpha, beta, 0, ws,
                                      ws_bytes, stream);
}

int kronq_accumulate_cov_limited(const void* A, int dtype, int64_t n_rows, int64_t d,
                                 int64_t lda, float* H, int64_t ldh, float alpha, float beta,
                                 int max_cus, void* ws, size_t ws_bytes, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(max_cus >= 0, KRONQ_ERR_INVALID_ARG, "max_cus must be >= 0");
  KQ_REQUIRE(valid_dtype(dtype), KRONQ_ERR_INVALID_ARG, "dtype must be KRONQ_BF16 or KRONQ_FP32");
  KQ_REQUIRE(H, KRONQ_ERR_INVALID_ARG, "H is NULL");
  KQ_REQUIRE(n_rows >= 0 && d >= 1 && d <= 65535, KRONQ_ERR_INVALID_ARG,
             "need n_rows >= 0 and 1 <= d <= 65535");
  KQ_REQUIRE(ldh >= d && aligned(H, 4), KRONQ_ERR_INVALID_ARG, "bad H leading dimension");
  if (n_rows > 0) {
    KQ_REQUIRE(A, KRONQ_ERR_INVALID_ARG, "A is NULL");
    KQ_REQUIRE(lda >= d, KRONQ_ERR_INVALID_ARG, "lda < d");
    if (dtype == KRONQ_BF16)
      KQ_REQUIRE(aligned(A, 16) && lda % 8 == 0, KRONQ_ERR_INVALID_ARG,
                 "bf16 A must be 16-byte aligned with lda divisible by 8");
    else
      KQ_REQUIRE(aligned(A, 4), KRONQ_ERR_INVALID_ARG, "fp32 A must be 4-byte aligned");
    KQ_TRY(check_ws(ws, ws_bytes, kq::cov_ws_bytes(dtype, n_rows, d)));
  }
  return kq::cov_launch(A, nullptr, dtype, n_rows, d, lda, H, ldh, alpha, beta, ws,
                        as_stream(stream), max_cus);
}

int kronq_cov_diag(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                   float* hdiag, int max_cus, void* ws, size_t ws_bytes, void* stream) {
  kq::clear_error();
  KQ_TRY(check_cov_diag_args(A, dtype, n_rows, d, lda, hdiag, max_cus));
  if (n_rows > 0) KQ_TRY(check_ws(ws, ws_bytes, kq::cov_diag_ws_bytes(n_rows, d)));
  return kq::cov_diag_launch(A, dtype, n_rows, d, lda, hdiag, max_cus, ws, as_stream(stream));
}

int kronq_cov_diag_noalloc(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                           float* hdiag, int max_cus, void* stream) {
  kq::clear_error();
  KQ_TRY(check_cov_diag_args(A, dtype, n_rows, d, lda, hdiag, max_cus));
  const size_t need = kq::cov_diag_need_bytes(n_rows, d, max_cus);
  KQ_REQUIRE(need <= size_t(KRONQ_NOALLOC_SCRATCH_BYTES), KRONQ_ERR_WORKSPACE,
             "kronq_cov_diag_noalloc: %zu bytes of partial sums needed (n_rows %lld, d %lld), "
             "the fixed scratch array holds %zu",
             need, (long long)n_rows, (long long)d, size_t(KRONQ_NOALLOC_SCRATCH_BYTES));
  void* scratch = nullptr;
  if (n_rows > 0) KQ_TRY(kq::cov_diag_scratch(as_stream(stream), &scratch));
  return kq::cov_diag_launch(A, dtype, n_rows, d, lda, hdiag, max_cus, scratch,
                             as_stream(stream));
}

int kronq_probe_mfma_bf16(const void* data, int iters, float* out, int64_t out_len,
                          int* workgroups, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(data && aligned(data, 16) && out && workgroups, KRONQ_ERR_INVALID_ARG,
             "data (16-byte aligned), out and workgroups are required");
  KQ_REQUIRE(iters >= 1, KRONQ_ERR_INVALID_ARG, "iters must be >= 1");
  int dev = 0, cus = 0;
  KQ_HIP(hipGetDevice(&dev));
  KQ_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  KQ_REQUIRE(out_len >= 2 * int64_t(cus), KRONQ_ERR_INVALID_ARG,
             "out holds %lld floats, %d needed", (long long)out_len, 2 * cus);
  return kq::mfma_peak_launch(static_cast<const uint16_t*>(data), iters, out, workgroups,
                              as_stream(stream));
}

int kronq_accumulate_cross(const void* A, const void* B, int dtype, int64_t n_rows, int64_t d,
                           int64_t ld, float* C, int64_t ldc, float alpha, float beta, void* ws,
                           size_t ws_bytes, void* stream) {
  return kronq_accumulate_cross_limited(A, B, dtype, n_rows, d, ld, C, ldc, alpha, beta, 0, ws,
                                        ws_bytes, stream);
}

int kronq_accumulate_cross_limited(const void* A, const void* B, int dtype, int64_t n_rows,
                                   int64_t d, int64_t ld, float* C, int64_t ldc, float alpha,
                                   float beta, int max_cus, void* ws, size_t ws_bytes,
                                   void* stream) {
  kq::clear_error();
  KQ_REQUIRE(max_cus >= 0, KRONQ_ERR_INVALID_ARG, "max_cus must be >= 0");
  KQ_REQUIRE(valid_dtype(dtype), KRONQ_ERR_INVALID_ARG, "dtype must be KRONQ_BF16 or KRONQ_FP32");
  KQ_REQUIRE(C, KRONQ_ERR_INVALID_ARG, "C is NULL");
  KQ_REQUIRE(n_rows >= 0 && d >= 1 && d <= 65535, KRONQ_ERR_INVALID_ARG,
             "need n_rows >= 0 and 1 <= d <= 65535");
  KQ_REQUIRE(ldc >= d && aligned(C, 4), KRONQ_ERR_INVALID_ARG, "bad C leading dimension");
  if (n_rows > 0) {
    KQ_REQUIRE(A && B, KRONQ_ERR_INVALID_ARG, "A or B is NULL");
    KQ_REQUIRE(ld >= d, KRONQ_ERR_INVALID_ARG, "ld < d");
    if (dtype == KRONQ_BF16)
      KQ_REQUIRE(aligned(A, 16) && aligned(B, 16) && ld % 8 == 0, KRONQ_ERR_INVALID_ARG,
                 "bf16 A and B must be 16-byte aligned with ld divisible by 8");
    else
      KQ_REQUIRE(aligned(A, 4) && aligned(B, 4), KRONQ_ERR_INVALID_ARG,
                 "fp32 A and B must be 4-byte aligned");
    KQ_TRY(check_ws(ws, ws_bytes, kq::cov_ws_bytes(dtype, n_rows, d, true)));
  }
  return kq::cov_launch(A, B, dtype, n_rows, d, ld, C, ldc, alpha, beta, ws, as_stream(stream),
                        max_cus);
}

int kronq_traces(const float* HX, int64_t d_in, int64_t ldx, const float* HG, int64_t d_out,
                 int64_t ldg, double* out3, void* stream) {
  kq::clear_error();
  KQ_REQUIRE((HX || HG) && out3, KRONQ_ERR_INVALID_ARG, "null pointer");
  KQ_REQUIRE((!HX || (d_in >= 1 && ldx >= d_in)) && (!HG || (d_out >= 1 && ldg >= d_out)),
             KRONQ_ERR_INVALID_ARG, "bad sizes");
  KQ_REQUIRE(aligned(out3, 8), KRONQ_ERR_INVALID_ARG, "out3 must be 8-byte aligned");
  return kq::traces_launch(HX, d_in, ldx, HG, d_out, ldg, out3, as_stream(stream));
}

int kronq_rotate(const void* W_in, int w_dtype, int64_t ldw_in, float* W, int64_t d_out,
                 int64_t d_in, int64_t ldw, float* HX, int64_t ldx, float* HG, int64_t ldg,
                 const int8_t* sign_in, const int8_t* sign_out, const float* q28_in,
                 const float* q28_out, float* sx, float* sg, int flags, void* ws,
                 size_t ws_bytes, void* stream) {
  kq::clear_error();
  const int known = KRONQ_BIIP | KRONQ_INVERSE | KRONQ_HX_ONLY | KRONQ_SX_GIVEN |
                    KRONQ_HG_DIAG | KRONQ_SG_GIVEN;
  KQ_REQUIRE((flags & ~known) == 0, KRONQ_ERR_INVALID_ARG, "unknown flag bits 0x%x",
             flags & ~known);
  const bool inv = flags & KRONQ_INVERSE;
  const bool hx_only = flags & KRONQ_HX_ONLY, sx_given = flags & KRONQ_SX_GIVEN;
  const bool hg_diag = flags & KRONQ_HG_DIAG, sg_given = flags & KRONQ_SG_GIVEN;
  KQ_REQUIRE(!(hx_only && sx_given) && !(inv && (hx_only || sx_given)), KRONQ_ERR_INVALID_ARG,
             "KRONQ_HX_ONLY, KRONQ_SX_GIVEN and KRONQ_INVERSE exclude each other");
  KQ_REQUIRE(!hg_diag || !(hx_only || sg_given || inv), KRONQ_ERR_INVALID_ARG,
             "KRONQ_HG_DIAG excludes KRONQ_HX_ONLY, KRONQ_SG_GIVEN and KRONQ_INVERSE");
  KQ_REQUIRE(!sg_given || sx_given, KRONQ_ERR_INVALID_ARG,
             "KRONQ_SG_GIVEN needs KRONQ_SX_GIVEN");
  if (!sg_given) {  // W_in is read (W_in is not touched by an H_G-only call)
    KQ_REQUIRE(W_in && valid_dtype(w_dtype), KRONQ_ERR_INVALID_ARG, "bad W_in");
    KQ_REQUIRE(ldw_in >= d_in, KRONQ_ERR_INVALID_ARG, "ldw_in < d_in");
    // W_in is read with 16-byte vector loads (8 bf16 or 4 fp32 values)
    KQ_REQUIRE(aligned(W_in, 16) && ldw_in % (w_dtype == KRONQ_BF16 ? 8 : 4) == 0,
               KRONQ_ERR_INVALID_ARG,
               "W_in must be 16-byte aligned with ldw_in divisible by 8 (bf16) or 4 (fp32)");
  }
  KQ_REQUIRE(d_out >= 1 && d_in >= 1, KRONQ_ERR_INVALID_ARG, "need d_out >= 1 and d_in >= 1");
  if (!hx_only && !sg_given) KQ_TRY(check_f32_mat(W, d_out, d_in, ldw, "W"));
  KQ_REQUIRE(sx && aligned(sx, 4) && (hx_only || (sg && aligned(sg, 4))), KRONQ_ERR_INVALID_ARG,
             "sx and sg are required");
  if (inv) {
    KQ_REQUIRE(w_dtype == KRONQ_FP32, KRONQ_ERR_INVALID_ARG, "KRONQ_INVERSE needs fp32 W_in");
    KQ_REQUIRE(ldw_in % 4 == 0 && aligned(W_in, 16), KRONQ_ERR_INVALID_ARG,
               "W_in must be 16-byte aligned with ldw_in divisible by 4");
  } else {
    if (!sx_given) KQ_TRY(check_f32_mat(HX, d_in, d_in, ldx, "HX"));
    if (hg_diag)
      KQ_REQUIRE(!HG || aligned(HG, 4), KRONQ_ERR_INVALID_ARG, "diag(H_G) misaligned");
    else if (HG && !hx_only)
      KQ_TRY(check_f32_mat(HG, d_out, d_out, ldg, "HG"));
    KQ_REQUIRE(HG || hx_only || !(flags & KRONQ_RESCALE_OUT), KRONQ_ERR_INVALID_ARG,
               "KRONQ_RESCALE_OUT needs H_G");
    KQ_REQUIRE(!sg_given || HG, KRONQ_ERR_INVALID_ARG, "KRONQ_SG_GIVEN needs H_G");
    KQ_REQUIRE(sg_given || W_in != static_cast<const void*>(W) || w_dtype == KRONQ_FP32,
               KRONQ_ERR_INVALID_ARG, "in-place rotation needs fp32 W");
  }
  if (flags & KRONQ_ROT_IN) KQ_TRY(check_rot_side(d_in, sign_in, q28_in, "input"));
  if ((flags & KRONQ_ROT_OUT) && !hx_only)
    KQ_TRY(check_rot_side(d_out, sign_out, q28_out, "output"));
  KQ_REQUIRE(d_in <= (int64_t(1) << 24) && d_out <= (int64_t(1) << 24), KRONQ_ERR_UNSUPPORTED,
             "dimension too large");
  KQ_TRY(check_ws(ws, ws_bytes, kq::rotate_ws_bytes(d_out, d_in)));
  return kq::rotate_launch(W_in, w_dtype, ldw_in, W, d_out, d_in, ldw, HX, ldx, HG, ldg, sign_in,
                           sign_out, q28_in, q28_out, sx, sg, flags, ws, as_stream(stream));
}

int kronq_rotate_drift(float* D, int64_t d_in, int64_t ldd, const float* sx,
                       const int8_t* sign_in, const float* q28_in, int flags, void* ws,
                       size_t ws_bytes, void* stream) {
  kq::clear_error();
  const int known = KRONQ_RESCALE_IN | KRONQ_ROT_IN;
  KQ_REQUIRE((flags & ~known) == 0, KRONQ_ERR_INVALID_ARG,
             "kronq_rotate_drift takes only KRONQ_RESCALE_IN and KRONQ_ROT_IN (0x%x given)",
             flags);
  KQ_TRY(check_f32_mat(D, d_in, d_in, ldd, "D"));
  KQ_REQUIRE(!(flags & KRONQ_RESCALE_IN) || (sx && aligned(sx, 4)), KRONQ_ERR_INVALID_ARG,
             "KRONQ_RESCALE_IN needs sx");
  if (flags & KRONQ_ROT_IN) KQ_TRY(check_rot_side(d_in, sign_in, q28_in, "input"));
  KQ_TRY(check_ws(ws, ws_bytes, kq::rotate_drift_ws_bytes(d_in)));
  return kq::rotate_drift_launch(D, d_in, ldd, sx, sign_in, q28_in, flags, ws, as_stream(stream));
}

int kronq_gptaq_correction(const float* D, int64_t d, int64_t ldd, const float* U, int64_t ldu,
                           float alpha, float* P, int64_t ldp, void* ws, size_t ws_bytes,
                           void* stream) {
  kq::clear_error();
  KQ_REQUIRE(d <= 65535, KRONQ_ERR_INVALID_ARG, "need d <= 65535");
  KQ_TRY(check_f32_mat(D, d, d, ldd, "D"));
  KQ_TRY(check_f32_mat(U, d, d, ldu, "U"));
  KQ_TRY(check_f32_mat(P, d, d, ldp, "P"));
  KQ_REQUIRE(static_cast<const float*>(P) != D && static_cast<const float*>(P) != U,
             KRONQ_ERR_INVALID_ARG, "P must not alias D or U");
  KQ_TRY(check_ws(ws, ws_bytes, kq::gptaq_ws_bytes(d)));
  return kq::gptaq_launch(D, d, ldd, U, ldu, alpha, P, ldp, ws, as_stream(stream));
}

int kronq_cholesky_inv(float* H, int64_t d, int64_t ldh, float damp_rel, float* Uout,
                       int64_t ldu, int* info, void* ws, size_t ws_bytes, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(H && Uout && info, KRONQ_ERR_INVALID_ARG, "null pointer");
  KQ_REQUIRE(d >= 1 && d <= 65535, KRONQ_ERR_INVALID_ARG, "need 1 <= d <= 65535");
  KQ_REQUIRE(ldh >= d && ldu >= d, KRONQ_ERR_INVALID_ARG, "bad leading dimension");
  KQ_REQUIRE(aligned(H, 4) && aligned(Uout, 4) && aligned(info, 4), KRONQ_ERR_INVALID_ARG,
             "misaligned pointer");
  KQ_REQUIRE(Uout != H, KRONQ_ERR_INVALID_ARG, "Uout must not alias H");
  KQ_REQUIRE(damp_rel >= 0.f, KRONQ_ERR_INVALID_ARG, "damp_rel must be >= 0");
  KQ_TRY(check_ws(ws, ws_bytes, kq::chol_ws_bytes(d)));
  return kq::chol_launch(H, d, ldh, damp_rel, Uout, ldu, info, ws, as_stream(stream));
}

int kronq_obs_quantize_layer(float* W, int64_t d_out, int64_t d_in, int64_t ldw,
                             const float* U, int64_t ldu, int bits, int group, int block,
                             uint8_t* codes, float* scales, float* zeros, float* err,
                             float* W_hat, void* ws, size_t ws_bytes, void* stream) {
  kq::clear_error();
  return obs_common(W, d_out, d_in, ldw, U, ldu, nullptr, 0, bits, group, block, codes, scales,
                    zeros, err, W_hat, ws, ws_bytes, stream);
}

int kronq_obs_quantize_layer_drift(float* W, int64_t d_out, int64_t d_in, int64_t ldw,
                                   const float* U, int64_t ldu, const float* P, int64_t ldp,
                                   int bits, int group, int block, uint8_t* codes, float* scales,
                                   float* zeros, float* err, float* W_hat, void* ws,
                                   size_t ws_bytes, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(P, KRONQ_ERR_INVALID_ARG, "P is NULL");
  return obs_common(W, d_out, d_in, ldw, U, ldu, P, ldp, bits, group, block, codes, scales, zeros,
                    err, W_hat, ws, ws_bytes, stream);
}

int kronq_pack_codes(const uint8_t* codes, int64_t d_out, int64_t d_in, int64_t ldq, int bits,
                     uint32_t* packed, int64_t ldp, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(bits == 2 || bits == 3 || bits == 4 || bits == 8, KRONQ_ERR_UNSUPPORTED,
             "bits must be 2, 3, 4 or 8");
  KQ_REQUIRE(codes && packed && aligned(packed, 4), KRONQ_ERR_INVALID_ARG, "bad pointer");
  KQ_REQUIRE(d_out >= 1 && d_in >= 32 && d_in % 32 == 0, KRONQ_ERR_SHAPE,
             "need d_out >= 1 and d_in a positive multiple of 32");
  KQ_REQUIRE(ldq >= d_in && ldp >= d_in * bits / 32, KRONQ_ERR_INVALID_ARG,
             "bad leading dimension");
  return kq::pack_codes_launch(codes, d_out, d_in, ldq, bits, packed, ldp, as_stream(stream));
}

int kronq_matrix_stats(const void* M, int dtype, int64_t rows, int64_t cols, int64_t ld,
                       double* out, void* ws, size_t ws_bytes, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(M && valid_dtype(dtype) && aligned(M, 4), KRONQ_ERR_INVALID_ARG,
             "M must be a 4-byte aligned KRONQ_BF16 or KRONQ_FP32 matrix");
  KQ_REQUIRE(rows >= 1 && cols >= 1 && ld >= cols && rows <= (int64_t(1) << 31) &&
                 cols <= (int64_t(1) << 31),
             KRONQ_ERR_INVALID_ARG, "bad sizes");
  KQ_REQUIRE(out && aligned(out, 8), KRONQ_ERR_INVALID_ARG, "out must be a double[5] device pointer");
  KQ_TRY(check_ws(ws, ws_bytes, kq::matrix_stats_ws_bytes(rows, cols)));
  return kq::matrix_stats_launch(M, dtype, rows, cols, ld, out, ws, as_stream(stream));
}

int kronq_eigh(const float* H, int64_t d, int64_t ldh, int sweeps, float* evals, float* Q,
               int64_t ldq, double* off, void* ws, size_t ws_bytes, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(d >= 1 && d <= 16384, KRONQ_ERR_UNSUPPORTED, "1 <= d <= 16384");
  KQ_REQUIRE(sweeps >= 1 && sweeps <= 64, KRONQ_ERR_INVALID_ARG, "1 <= sweeps <= 64");
  KQ_REQUIRE(H && aligned(H, 4) && ldh >= d, KRONQ_ERR_INVALID_ARG, "bad H");
  KQ_REQUIRE(Q && aligned(Q, 4) && ldq >= d, KRONQ_ERR_INVALID_ARG, "bad Q");
  KQ_REQUIRE(evals && aligned(evals, 4) && off && aligned(off, 8), KRONQ_ERR_INVALID_ARG,
             "evals and off are required");
  const char *h0 = reinterpret_cast<const char*>(H), *q0 = reinterpret_cast<const char*>(Q);
  const size_t hb = (size_t(d - 1) * size_t(ldh) + size_t(d)) * 4;
  const size_t qb = (size_t(d - 1) * size_t(ldq) + size_t(d)) * 4;
  KQ_REQUIRE(q0 + qb <= h0 || h0 + hb <= q0, KRONQ_ERR_INVALID_ARG, "Q must not overlap H");
  KQ_TRY(check_ws(ws, ws_bytes, kq::eigh_ws_bytes(d)));
  return kq::eigh_launch(H, d, ldh, sweeps, evals, Q, ldq, off, ws, as_stream(stream));
}

int kronq_proxy_loss_factors(const float* HG, int64_t d_out, int64_t ldg, const void* W,
                             int w_dtype, int64_t ldw, int64_t d_in, const float* Hd, int64_t ldh,
                             const float* U, int64_t ldu, const double* alphas, int n_alpha,
                             double* out, void* ws, size_t ws_bytes, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(d_out >= 1 && d_in >= 1 && d_out <= (int64_t(1) << 31) && d_in <= (int64_t(1) << 31),
             KRONQ_ERR_INVALID_ARG, "bad sizes");
  KQ_REQUIRE(HG && aligned(HG, 4) && ldg >= d_out, KRONQ_ERR_INVALID_ARG, "bad H_G");
  KQ_REQUIRE(W && valid_dtype(w_dtype) && aligned(W, 4) && ldw >= d_in, KRONQ_ERR_INVALID_ARG,
             "bad W");
  KQ_REQUIRE(Hd && aligned(Hd, 4) && ldh >= d_in, KRONQ_ERR_INVALID_ARG, "bad H~");
  KQ_REQUIRE(U && aligned(U, 4) && ldu >= d_in, KRONQ_ERR_INVALID_ARG, "bad U");
  KQ_REQUIRE(n_alpha >= 0 && n_alpha <= KRONQ_MAX_ALPHAS && (n_alpha == 0 || alphas),
             KRONQ_ERR_INVALID_ARG, "0 <= n_alpha <= %d host exponents", KRONQ_MAX_ALPHAS);
  KQ_REQUIRE(out && aligned(out, 8), KRONQ_ERR_INVALID_ARG, "out is required");
  KQ_TRY(check_ws(ws, ws_bytes, kq::proxy_ws_bytes(d_out, d_in)));
  return kq::proxy_launch(HG, ldg, W, w_dtype, ldw, d_out, d_in, Hd, ldh, U, ldu, alphas,
                          n_alpha, out, ws, as_stream(stream));
}

int kronq_online_factors(const float* s, const int8_t* sign, int64_t d, float* mul, void* stream) {
  kq::clear_error();
  KQ_REQUIRE(d >= 1 && mul && aligned(mul, 16), KRONQ_ERR_INVALID_ARG,
             "mul must be a 16-byte aligned device pointer and d >= 1");
  KQ_REQUIRE(!s || aligned(s, 4), KRONQ_ERR_INVALID_ARG, "misaligned s");
  return kq::inverse_multipliers(s, sign, d, mul, as_stream(stream));
}

int kronq_online_matvec(const uint32_t* packed, int64_t ldp, const float* scales,
                        const float* zeros, int64_t ldsz, int bits, int group, int64_t d_out,
                        int64_t d_in, const float* mul_in, const float* mul_out,
                        const float* q28_in, const float* q28_out, int flags, const void* x,
                        int x_dtype, int64_t ldx, int64_t batch, float* y, int64_t ldy, void* ws,
                        size_t ws_bytes, void* stream) {
  kq::clear_error();
  KQ_REQUIRE((flags & ~KRONQ_BIIP) == 0, KRONQ_ERR_INVALID_ARG, "unknown flag bits 0x%x",
             flags & ~KRONQ_BIIP);
  KQ_REQUIRE(bits == 2 || bits == 3 || bits == 4 || bits == 8, KRONQ_ERR_UNSUPPORTED,
             "bits must be 2, 3, 4 or 8");
  KQ_REQUIRE(d_out >= 1 && d_in >= 128 && d_out <= (int64_t(1) << 24), KRONQ_ERR_INVALID_ARG,
             "bad sizes");
  KQ_REQUIRE(group >= 128 && group % 128 == 0 && d_in % group == 0, KRONQ_ERR_SHAPE,
             "group must be a multiple of 128 dividing d_in");
  KQ_REQUIRE(batch >= 1 && batch <= 4 && batch * d_in <= 32768, KRONQ_ERR_UNSUPPORTED,
             "1 <= batch <= 4 and batch * d_in <= 32768 (the activations are held in LDS)");
  KQ_REQUIRE(packed && aligned(packed, 16) && ldp % 4 == 0 && ldp >= d_in * bits / 32,
             KRONQ_ERR_INVALID_ARG,
             "packed must be 16-byte aligned with ldp >= d_in * bits / 32, divisible by 4");
  KQ_REQUIRE(scales && zeros && aligned(scales, 4) && aligned(zeros, 4) && ldsz >= d_in / group,
             KRONQ_ERR_INVALID_ARG, "bad scales or zeros");
  KQ_REQUIRE(!mul_in || aligned(mul_in, 16), KRONQ_ERR_INVALID_ARG, "mul_in must be 16-byte aligned");
  KQ_REQUIRE(!mul_out || aligned(mul_out, 16), KRONQ_ERR_INVALID_ARG,
             "mul_out must be 16-byte aligned");
  KQ_REQUIRE(x && valid_dtype(x_dtype) && ldx >= d_in && aligned(x, 16) &&
                 ldx % (x_dtype == KRONQ_BF16 ? 8 : 4) == 0,
             KRONQ_ERR_INVALID_ARG,
             "x must be 16-byte aligned with ldx divisible by 8 (bf16) or 4 (fp32)");
  KQ_REQUIRE(y && aligned(y, 16) && ldy >= d_out && ldy % 4 == 0, KRONQ_ERR_INVALID_ARG,
             "y must be 16-byte aligned with ldy >= d_out divisible by 4");
  if (flags & KRONQ_ROT_IN) {
    const kq::RotDim r = kq::rot_dim(d_in);
    KQ_REQUIRE(r.ok && d_in <= kMaxRotDim, KRONQ_ERR_UNSUPPORTED,
               "input dimension %lld is not 2^k or 28*2^k", (long long)d_in);
    KQ_REQUIRE(!r.has28 || (q28_in && aligned(q28_in, 4)), KRONQ_ERR_INVALID_ARG,
               "input dimension 28 * 2^k needs the 28 x 28 factor");
  }
  if (flags & KRONQ_ROT_OUT) {
    const kq::RotDim r = kq::rot_dim(d_out);
    KQ_REQUIRE(r.ok && d_out <= kMaxRotDim, KRONQ_ERR_UNSUPPORTED,
               "output dimension %lld is not 2^k or 28*2^k", (long long)d_out);
    KQ_REQUIRE(!r.has28 || (q28_out && aligned(q28_out, 4)), KRONQ_ERR_INVALID_ARG,
               "output dimension 28 * 2^k needs the 28 x 28 factor");
  }
  KQ_REQUIRE(d_out <= kMaxRotDim, KRONQ_ERR_UNSUPPORTED,
             "d_out > %lld: an output vector must fit the LDS", (long long)kMaxRotDim);
  KQ_TRY(check_ws(ws, ws_bytes, kq::online_ws_bytes(d_out, d_in, batch)));
  return kq::online_matvec_launch(packed, ldp, scales, zeros, ldsz, bits, group, d_out, d_in,
                                  mul_in, mul_out, q28_in, q28_out, flags, x, x_dtype, ldx, batch,
                                  y, ldy, ws, as_stream(stream));
}

int kronq_layer_loss(const void* W, int w_dtype, int64_t ldw, const float* W_hat,
                     int64_t ldwh, int64_t d_out, int64_t d_in, const float* HX, int64_t ldx,
                     const float* HG, int64_t ldg, double* loss, void* ws, size_t ws_bytes,
                     void* stream) {
  kq::clear_error();
  KQ_REQUIRE(W && valid_dtype(w_dtype) && loss, KRONQ_ERR_INVALID_ARG, "bad W or loss");
  KQ_REQUIRE(d_out >= 1 && d_in >= 1 && d_out <= 65535 && ldw >= d_in, KRONQ_ERR_INVALID_ARG,
             "bad sizes");
  KQ_REQUIRE(aligned(W, w_dtype == KRONQ_BF16 ? 2 : 4) && aligned(loss, 8), KRONQ_ERR_INVALID_ARG,
             "misaligned pointer");
  KQ_REQUIRE(!W_hat || (ldwh >= d_in && aligned(W_hat, 4)), KRONQ_ERR_INVALID_ARG, "bad W_hat");
  KQ_TRY(check_f32_mat(HX, d_in, d_in, ldx, "HX"));
  KQ_TRY(check_f32_mat(HG, d_out, d_out, ldg, "HG"));
  KQ_TRY(check_ws(ws, ws_bytes, kq::loss_ws_bytes(d_out, d_in)));
  return kq::loss_launch(W, w_dtype, ldw, W_hat, ldwh, d_out, d_in, HX, ldx, HG, ldg, loss, ws,
                         as_stream(stream));
}

}  // extern "C"
