// Lazy-block column-wise OBS with group quantisation (eq. obs_update, Prop. 1 with the drift
// correction P = 0; Alg. 2).
//
// Per block of 128 columns (= one quantisation group):
//   * sweep kernel: rows are independent given U, so each row is one 16-lane group of a wave
//     (4 rows per wave, 16 rows per workgroup) and each lane keeps 8 consecutive columns of the
//     block in registers. Column j: the owning lane quantises it and forms the scaled error
//     e_j = (w_j - w_hat_j) / U_jj, one DPP row broadcast hands e_j to the other 15 lanes, and
//     every lane applies it to its 8 columns with U[j, its columns] read from the workgroup's
//     LDS copy of the 128 x 128 block of U (upper triangular, so columns already done are left
//     alone). Group parameters come from the row's 128 values at the start of the block.
//     Codes, errors and dequantised values are written from registers at the end.
//   * trailing updates, lazily in two levels: after each block, W[:, rest of its group of 4
//     blocks] -= E_b U[b, rest of group] (K = 128); after the last block of a group,
//     W[:, beyond the group] -= E_group U[group, beyond] (K = 512). Every column still receives
//     the update of every earlier block before it is swept, as in the one-level scheme, with a
//     quarter of the passes over W. Both products run on the bf16 matrix cores with the
//     fp32-accurate three-term split (gemm_bf16x3.hip); U^T is split once per layer.
// The quantiser (reading of the paper's "quant"): xmin = min(0, min w), xmax = max(0, max w),
// (-1, 1) when both are 0; scale = float32((xmax - xmin) / (2^b - 1)) in float64;
// zero = rint(-xmin / scale); q = clamp(rint(w / scale) + zero, 0, 2^b - 1);
// w_hat = float32(scale * (q - zero)). The code must be the one of the exact quotient w / scale
// rounded half to even: the kernel forms t = w * (1 / scale) in fp32 (relative error below
// 2.4e-7) and takes rint(t) unless t lies within 1e-6 (|t| + 1) of a half-integer, where it
// falls back to the IEEE float64 division. w_hat in fp32 equals the float64 form exactly
// (scale and q - zero are exact fp32 operands of one correctly rounded product).
#include <utility>

#include "kq_common.hpp"

namespace kq {
namespace {

constexpr int OB = 128;          // block = group
constexpr int LPR = 16;          // lanes per row
constexpr int CPL = OB / LPR;    // columns per lane
constexpr int RPW = 64 / LPR;    // rows per wave
constexpr int RPG = 4 * RPW;     // rows per workgroup (4 waves)
constexpr int GRP = 4;           // blocks per group of the two-level lazy update

// v broadcast from lane `src` of each 16-lane row to the whole row (DPP row_newbcast)
template <int src>
__device__ __forceinline__ float row_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x150 + src, 0xF, 0xF,
                                                    false));
}

// one column of the sweep: j = 8 * OWN + S (compile-time)
template <int OWN, int S>
__device__ __forceinline__ void sweep_col(float (&w)[CPL], float (&ev)[CPL], uint32_t (&qc)[CPL],
                                          const float* ub, const float* rinv, int sub, int cb,
                                          float scale, float inv_s, double dscale, float fzero,
                                          float fmaxq) {
  constexpr int j = OWN * CPL + S;
  const float x = w[S];
  const float t = x * inv_s;
  float qf = __builtin_rintf(t);
  const bool tie = fabsf(t - floorf(t) - 0.5f) <= 1e-6f * (fabsf(t) + 1.f);
  if (tie && sub == OWN) qf = float(__builtin_rint(double(x) / dscale));
  const float q = fminf(fmaxf(qf + fzero, 0.f), fmaxq);
  const float wh = scale * (q - fzero);
  const float e = (x - wh) * rinv[j];
  if (sub == OWN) {
    ev[S] = e;
    qc[S] = uint32_t(q);
  }
  const float eb = row_bcast<OWN>(e);
  const float4 u0 = *reinterpret_cast<const float4*>(ub + j * OB + cb);
  const float4 u1 = *reinterpret_cast<const float4*>(ub + j * OB + cb + 4);
  w[0] = fmaf(-eb, u0.x, w[0]);
  w[1] = fmaf(-eb, u0.y, w[1]);
  w[2] = fmaf(-eb, u0.z, w[2]);
  w[3] = fmaf(-eb, u0.w, w[3]);
  w[4] = fmaf(-eb, u1.x, w[4]);
  w[5] = fmaf(-eb, u1.y, w[5]);
  w[6] = fmaf(-eb, u1.z, w[6]);
  w[7] = fmaf(-eb, u1.w, w[7]);
}

template <int OWN>
__device__ __forceinline__ void sweep_lane_cols(float (&w)[CPL], float (&ev)[CPL],
                                                uint32_t (&qc)[CPL], const float* ub,
                                                const float* rinv, int sub, int cb, float scale,
                                                float inv_s, double dscale, float fzero,
                                                float fmaxq) {
  sweep_col<OWN, 0>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq);
  sweep_col<OWN, 1>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq);
  sweep_col<OWN, 2>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq);
  sweep_col<OWN, 3>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq);
  sweep_col<OWN, 4>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq);
  sweep_col<OWN, 5>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq);
  sweep_col<OWN, 6>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq);
  sweep_col<OWN, 7>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq);
}

template <int... OWN>
__device__ __forceinline__ void sweep_all(std::integer_sequence<int, OWN...>, float (&w)[CPL],
                                          float (&ev)[CPL], uint32_t (&qc)[CPL], const float* ub,
                                          const float* rinv, int sub, int cb, float scale,
                                          float inv_s, double dscale, float fzero, float fmaxq) {
  (sweep_lane_cols<OWN>(w, ev, qc, ub, rinv, sub, cb, scale, inv_s, dscale, fzero, fmaxq), ...);
}

__global__ __launch_bounds__(256) void obs_sweep(float* __restrict__ W, int64_t d_out,
                                                 int64_t ldw, const float* __restrict__ U,
                                                 int64_t ldu, int64_t c0, int bits,
                                                 uint8_t* __restrict__ codes, int64_t ldq,
                                                 float* __restrict__ scales,
                                                 float* __restrict__ zeros, int64_t ldsz,
                                                 int64_t blk, float* __restrict__ E, int64_t lde,
                                                 float* __restrict__ W_hat, int64_t ldwh) {
  __shared__ __attribute__((aligned(16))) float ub[OB * OB];  // U[c0 + j][c0 + k]
  __shared__ float rinv[OB];                                   // 1 / U_jj
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane & (LPR - 1), cb = sub * CPL;
  const int64_t row = int64_t(blockIdx.x) * RPG + wave * RPW + (lane >> 4);
  const bool live = row < d_out;
  const int64_t rr = live ? row : d_out - 1;  // rows past the end recompute the last row

  for (int idx = tid; idx < OB * OB / 4; idx += 256) {
    const int j = idx / (OB / 4), k4 = (idx % (OB / 4)) * 4;
    *reinterpret_cast<float4*>(ub + j * OB + k4) =
        *reinterpret_cast<const float4*>(U + (c0 + j) * ldu + c0 + k4);
  }
  if (tid < OB) rinv[tid] = 1.f / U[(c0 + tid) * ldu + c0 + tid];
  float w[CPL];
  {
    const float4 a = *reinterpret_cast<const float4*>(W + rr * ldw + c0 + cb);
    const float4 b = *reinterpret_cast<const float4*>(W + rr * ldw + c0 + cb + 4);
    w[0] = a.x, w[1] = a.y, w[2] = a.z, w[3] = a.w, w[4] = b.x, w[5] = b.y, w[6] = b.z, w[7] = b.w;
  }
  // group parameters from the row's current 128 values (group start = block start)
  float xmin = 0.f, xmax = 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    xmin = fminf(xmin, w[c]);
    xmax = fmaxf(xmax, w[c]);
  }
#pragma unroll
  for (int o = 1; o < LPR; o <<= 1) {
    xmin = fminf(xmin, __shfl_xor(xmin, o, LPR));
    xmax = fmaxf(xmax, __shfl_xor(xmax, o, LPR));
  }
  if (xmax == xmin) {
    xmin = -1.f;
    xmax = 1.f;
  }
  const double maxq = double((1 << bits) - 1);
  const float scale = float((double(xmax) - double(xmin)) / maxq);
  const double zero = __builtin_rint(-double(xmin) / double(scale));
  const float fzero = float(zero), inv_s = 1.f / scale;
  __syncthreads();

  float ev[CPL];
  uint32_t qc[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) ev[c] = 0.f, qc[c] = 0u;
  sweep_all(std::make_integer_sequence<int, LPR>{}, w, ev, qc, ub, rinv, sub, cb, scale, inv_s,
            double(scale), fzero, float(maxq));

  if (!live) return;
  if (sub == 0) {
    scales[row * ldsz + blk] = scale;
    zeros[row * ldsz + blk] = fzero;
  }
  float wh[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) wh[c] = scale * (float(qc[c]) - fzero);
  const float4 h0 = make_float4(wh[0], wh[1], wh[2], wh[3]);
  const float4 h1 = make_float4(wh[4], wh[5], wh[6], wh[7]);
  *reinterpret_cast<float4*>(W + row * ldw + c0 + cb) = h0;
  *reinterpret_cast<float4*>(W + row * ldw + c0 + cb + 4) = h1;
  if (W_hat) {
    *reinterpret_cast<float4*>(W_hat + row * ldwh + c0 + cb) = h0;
    *reinterpret_cast<float4*>(W_hat + row * ldwh + c0 + cb + 4) = h1;
  }
  *reinterpret_cast<float4*>(E + row * lde + cb) = make_float4(ev[0], ev[1], ev[2], ev[3]);
  *reinterpret_cast<float4*>(E + row * lde + cb + 4) = make_float4(ev[4], ev[5], ev[6], ev[7]);
  uint2 pk;
  pk.x = qc[0] | (qc[1] << 8) | (qc[2] << 16) | (qc[3] << 24);
  pk.y = qc[4] | (qc[5] << 8) | (qc[6] << 16) | (qc[7] << 24);
  *reinterpret_cast<uint2*>(codes + row * ldq + c0 + cb) = pk;
}

}  // namespace

size_t obs_ws_bytes(int64_t d_out, int64_t d_in) {
  if (d_out <= 0 || d_in <= 0) return 0;
  return align256(size_t(d_out) * GRP * OB * sizeof(float)) +
         2 * align256(size_t(d_in) * size_t(d_in) * sizeof(uint16_t)) + 256;
}

int obs_launch(float* W, int64_t d_out, int64_t d_in, int64_t ldw, const float* U, int64_t ldu,
               int bits, uint8_t* codes, float* scales, float* zeros, float* err, float* W_hat,
               void* ws, hipStream_t s) {
  const int64_t nblk = d_in / OB;
  const unsigned grid = unsigned(cdiv(d_out, RPG));
  Carver cv(ws);
  float* Ews = cv.take<float>(size_t(d_out) * GRP * OB);
  uint16_t* Uth = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  uint16_t* Utl = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  // U^T split once into bf16 high and low parts: the B operand of the trailing updates
  KQ_TRY(split_transpose_launch(U, ldu, d_in, Uth, Utl, d_in, s));
  for (int64_t g0 = 0; g0 < nblk; g0 += GRP) {
    const int64_t gend = g0 + GRP < nblk ? g0 + GRP : nblk;
    // errors of this group's blocks: the caller's err (ld d_in) or the workspace (ld GRP * OB)
    float* Eg = err ? err + g0 * OB : Ews;
    const int64_t lde = err ? d_in : GRP * OB;
    for (int64_t b = g0; b < gend; ++b) {
      const int64_t c0 = b * OB;
      float* Eb = Eg + (b - g0) * OB;
      KQ_TRY(launch("obs_sweep", obs_sweep, dim3(grid), dim3(256), 0, s, W, d_out, ldw, U, ldu,
                    c0, bits, codes, d_in, scales, zeros, nblk, b, Eb, lde, W_hat, d_in));
      const int64_t near = (gend - b - 1) * OB;  // rest of the group
      if (near > 0)  // W[:, c0+OB : gend*OB] -= E_b U[c0 : c0+OB, c0+OB : gend*OB]
        KQ_TRY(gemm_bf16x3_sub(d_out, near, OB, Eb, lde, Uth + (c0 + OB) * d_in + c0,
                               Utl + (c0 + OB) * d_in + c0, d_in, W + c0 + OB, ldw, s,
                               "obs_trailing_update"));
    }
    const int64_t rem = d_in - gend * OB;  // beyond the group
    if (rem > 0)  // W[:, gend*OB :] -= E_group U[g0*OB : gend*OB, gend*OB :]
      KQ_TRY(gemm_bf16x3_sub(d_out, rem, (gend - g0) * OB, Eg, lde,
                             Uth + gend * OB * d_in + g0 * OB, Utl + gend * OB * d_in + g0 * OB,
                             d_in, W + gend * OB, ldw, s, "obs_trailing_update"));
  }
  return KRONQ_OK;
}

}  // namespace kq
