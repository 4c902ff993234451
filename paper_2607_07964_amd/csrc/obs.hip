// Lazy-block column-wise OBS with group quantisation (eq. obs_update, Prop. 1 with the drift
// correction P = 0; Alg. 2).
//
// Per block of 128 columns (= one quantisation group):
//   * sweep kernel, one wave per 64 rows, one row per lane (rows are independent given U):
//     the W block is staged column-major in LDS (lane r touches column c at a conflict-free
//     address), the 128 x 128 block of U in LDS (every U read is a broadcast). Group
//     parameters come from the row's current 128 values. Columns are processed in sub-blocks
//     of 8 held in registers: quantise, scaled error e_j = (w_j - w_hat_j) / U_jj, update the
//     remaining sub-block columns in registers, then apply the 8 errors to the rest of the
//     block (8 FMAs per LDS read/write). The error replaces the column in LDS; codes stay in
//     LDS and everything is written back coalesced at the end, the dequantised values being
//     recomputed from code, scale and zero with the same operations.
//   * trailing update W[:, blk_end:] -= E U[blk, blk_end:] on the fp32 MFMA GEMM (K = 128).
// The quantiser (reading of the paper's "quant"): xmin = min(0, min w), xmax = max(0, max w),
// (-1, 1) when both are 0; scale = float32((xmax - xmin) / (2^b - 1)) in float64;
// zero = rint(-xmin / scale); q = clamp(rint(w / scale) + zero, 0, 2^b - 1);
// w_hat = float32(scale * (q - zero)). Divisions are IEEE float64 (no reciprocal), rint rounds
// half to even, so a code depends only on (w, scale).
#include "kq_common.hpp"

namespace kq {
namespace {

constexpr int OB = 128;       // block = group
constexpr int OR = 64;        // rows per workgroup (one wave)
constexpr int WLD = OR + 1;   // LDS stride of a W-block column
constexpr int SB = 8;         // columns per register sub-block

__device__ __forceinline__ float dequant(float scale, double zero, double q) {
  return float(double(scale) * (q - zero));
}

__global__ __launch_bounds__(OR) void obs_sweep(float* __restrict__ W, int64_t d_out, int64_t ldw,
                                                const float* __restrict__ U, int64_t ldu,
                                                int64_t c0, int bits, uint8_t* __restrict__ codes,
                                                int64_t ldq, float* __restrict__ scales,
                                                float* __restrict__ zeros, int64_t ldsz,
                                                int64_t blk, float* __restrict__ E, int64_t lde,
                                                float* __restrict__ W_hat, int64_t ldwh) {
  __shared__ float wb[OB * WLD];   // wb[c * WLD + r]
  __shared__ float ub[OB * OB];    // ub[j * OB + k] = U[c0 + j][c0 + k]
  __shared__ uint32_t qb[OR * OB / 4];
  __shared__ float sc[OR];
  __shared__ double zr[OR];
  const int lane = threadIdx.x;
  const int64_t r0 = int64_t(blockIdx.x) * OR;
  const double maxq = double((1 << bits) - 1);

  for (int idx = lane; idx < OB * OB / 4; idx += OR) {
    const int j = idx / (OB / 4), k4 = (idx % (OB / 4)) * 4;
    *reinterpret_cast<float4*>(ub + j * OB + k4) =
        *reinterpret_cast<const float4*>(U + (c0 + j) * ldu + c0 + k4);
  }
  for (int idx = lane; idx < OR * OB / 4; idx += OR) {
    const int r = idx / (OB / 4), c4 = (idx % (OB / 4)) * 4;
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r0 + r < d_out) x = *reinterpret_cast<const float4*>(W + (r0 + r) * ldw + c0 + c4);
    wb[(c4 + 0) * WLD + r] = x.x;
    wb[(c4 + 1) * WLD + r] = x.y;
    wb[(c4 + 2) * WLD + r] = x.z;
    wb[(c4 + 3) * WLD + r] = x.w;
  }
  __syncthreads();

  // group parameters from the current W (group start = block start)
  float xmin = 0.f, xmax = 0.f;
  for (int c = 0; c < OB; ++c) {
    const float v = wb[c * WLD + lane];
    xmin = fminf(xmin, v);
    xmax = fmaxf(xmax, v);
  }
  if (xmax == xmin) {
    xmin = -1.f;
    xmax = 1.f;
  }
  const float scale = float((double(xmax) - double(xmin)) / maxq);
  const double zero = __builtin_rint(-double(xmin) / double(scale));
  sc[lane] = scale;
  zr[lane] = zero;
  if (r0 + lane < d_out) {
    scales[(r0 + lane) * ldsz + blk] = scale;
    zeros[(r0 + lane) * ldsz + blk] = float(zero);
  }
  uint8_t* qrow = reinterpret_cast<uint8_t*>(qb) + lane * OB;

  for (int j0 = 0; j0 < OB; j0 += SB) {
    float w[SB], e[SB];
#pragma unroll
    for (int jj = 0; jj < SB; ++jj) w[jj] = wb[(j0 + jj) * WLD + lane];
#pragma unroll
    for (int jj = 0; jj < SB; ++jj) {
      double q = __builtin_rint(double(w[jj]) / double(scale)) + zero;
      q = q < 0.0 ? 0.0 : (q > maxq ? maxq : q);
      const float wh = dequant(scale, zero, q);
      const float ej = (w[jj] - wh) / ub[(j0 + jj) * OB + j0 + jj];
      e[jj] = ej;
      qrow[j0 + jj] = uint8_t(q);
#pragma unroll
      for (int kk = jj + 1; kk < SB; ++kk) w[kk] = fmaf(-ej, ub[(j0 + jj) * OB + j0 + kk], w[kk]);
    }
#pragma unroll
    for (int jj = 0; jj < SB; ++jj) wb[(j0 + jj) * WLD + lane] = e[jj];
    for (int k = j0 + SB; k < OB; ++k) {
      float acc = wb[k * WLD + lane];
#pragma unroll
      for (int jj = 0; jj < SB; ++jj) acc = fmaf(-e[jj], ub[(j0 + jj) * OB + k], acc);
      wb[k * WLD + lane] = acc;
    }
  }
  __syncthreads();

  // write back: errors, dequantised values (W and W_hat), codes
  for (int idx = lane; idx < OR * OB / 4; idx += OR) {
    const int r = idx / (OB / 4), c4 = (idx % (OB / 4)) * 4;
    const int64_t gr = r0 + r;
    if (gr >= d_out) continue;
    const float4 ev = make_float4(wb[(c4 + 0) * WLD + r], wb[(c4 + 1) * WLD + r],
                                  wb[(c4 + 2) * WLD + r], wb[(c4 + 3) * WLD + r]);
    *reinterpret_cast<float4*>(E + gr * lde + c4) = ev;
    const uint32_t qw = qb[r * (OB / 4) + c4 / 4];
    const float s = sc[r];
    const double z = zr[r];
    const float4 hv = make_float4(dequant(s, z, double(qw & 0xFF)), dequant(s, z, double((qw >> 8) & 0xFF)),
                                  dequant(s, z, double((qw >> 16) & 0xFF)), dequant(s, z, double(qw >> 24)));
    *reinterpret_cast<float4*>(W + gr * ldw + c0 + c4) = hv;
    if (W_hat) *reinterpret_cast<float4*>(W_hat + gr * ldwh + c0 + c4) = hv;
    *reinterpret_cast<uint32_t*>(codes + gr * ldq + c0 + c4) = qw;
  }
}

}  // namespace

size_t obs_ws_bytes(int64_t d_out, int64_t d_in) {
  if (d_out <= 0 || d_in <= 0) return 0;
  return align256(size_t(d_out) * OB * sizeof(float)) + 256;
}

int obs_launch(float* W, int64_t d_out, int64_t d_in, int64_t ldw, const float* U, int64_t ldu,
               int bits, uint8_t* codes, float* scales, float* zeros, float* err, float* W_hat,
               void* ws, hipStream_t s) {
  const int64_t nblk = d_in / OB;
  const unsigned grid = unsigned(cdiv(d_out, OR));
  for (int64_t b = 0; b < nblk; ++b) {
    const int64_t c0 = b * OB;
    float* E = err ? err + c0 : static_cast<float*>(ws);
    const int64_t lde = err ? d_in : OB;
    KQ_TRY(launch("obs_sweep", obs_sweep, dim3(grid), dim3(OR), 0, s, W, d_out, ldw, U, ldu, c0,
                  bits, codes, d_in, scales, zeros, nblk, b, E, lde, W_hat ? W_hat : nullptr,
                  d_in));
    const int64_t rem = d_in - c0 - OB;
    if (rem > 0)
      KQ_TRY(gemm_f32(0, d_out, rem, OB, -1.f, E, lde, U + c0 * ldu + c0 + OB, ldu, 1.f,
                      W + c0 + OB, ldw, s, "obs_trailing_update"));
  }
  return KRONQ_OK;
}

}  // namespace kq
