// Lazy-block column-wise OBS with group quantisation (eq. obs_update; Prop. 1 eq. kronq_update
// with or without the drift correction P; Alg. 2).
//
// Per block of 128 columns:
//   * sweep kernel: rows are independent given U, so each row is one 8-lane group of a wave
//     (8 rows per wave, 32 rows per workgroup; with the drift correction 16-lane groups) and
//     each lane keeps 16 (8) consecutive columns of the block in registers. Column j: the
//     owning lane quantises it and forms the scaled error e_j = (w_j - w_hat_j) / U_jj, a DPP
//     broadcast (two for 8-lane groups, one per half of a 16-lane DPP row) hands e_j to the
//     rest of the group, and every lane applies it to its columns with U[j, its columns] read from the workgroup's
//     LDS copy of the 128 x 128 block of U (upper triangular, so columns already done are left
//     alone). With the drift correction a second broadcast hands out w_j as it stood before
//     quantisation and every lane adds w_j P[j, its columns] from an LDS copy of the block of P
//     (strictly upper). Codes, errors, the pre-quantisation values (drift) and dequantised
//     values are written from registers at the end.
//   * group parameters: a group of 128 columns takes them from the row's 128 values at the
//     start of its block, inside the sweep kernel; a wider group (256, ..., d_in: the paper's
//     per-channel grid is group = d_in) takes them from the row's current values over the whole
//     group, in a reduction kernel launched when the sweep reaches the group's first block.
//   * trailing updates, lazily in two levels: after each block, W[:, rest of its lazy group of
//     (up to) 4 blocks] -= E_b U[b, rest of group] (K = 128); after the last block of a lazy
//     group, W[:, beyond] -= E_group U[group, beyond] (K = 512). With the drift correction the
//     same passes also add W_b P[b, ...], as a second K range of the same product. Every column
//     receives the update of every earlier block before it is swept, as in the one-level scheme,
//     with a quarter of the passes over W. The lazy group is shortened when needed so that a
//     wide quantisation group lies inside one lazy group or starts one (its columns are then
//     current when its parameters are taken). The products run on the bf16 matrix cores with
//     the fp32-accurate three-term split (gemm_bf16x3.hip); U^T and -P^T are split once per
//     layer.
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

constexpr int OB = 128;          // block (and the smallest group)
// Lanes per row of the sweep kernel: 8 (16 columns per lane) without the drift correction, 16
// (8 columns per lane) with it, whose second broadcast and P block would not fit the registers
// of 16 columns. 8 lanes halve the instructions per row: beside the H_G covariance, two waves
// per SIMD, the sweep's 32 blocks at q_proj take 2.75 ms instead of 3.2 ms (alone 1.8 against
// 1.67 ms).
template <bool DRIFT>
struct SweepLayout {
  static constexpr int LPR = DRIFT ? 16 : 8;  // lanes per row
  static constexpr int CPL = OB / LPR;        // columns per lane
  static constexpr int RPW = 64 / LPR;        // rows per wave
  static constexpr int RPG = 4 * RPW;         // rows per workgroup (4 waves)
};
constexpr int GRP = 4;           // blocks per group of the two-level lazy update (at most)

// v broadcast from lane `src` of each LPR-lane row group to the whole group (DPP row_newbcast
// over a 16-lane DPP row; for 8-lane groups one per half of it, selected by the bank mask)
template <int LPR, int src>
__device__ __forceinline__ float row_bcast(float v) {
  const int x = __float_as_int(v);
  if constexpr (LPR == 16) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0x150 + src, 0xF, 0xF, false));
  } else {
    static_assert(LPR == 8, "row groups of 8 or 16 lanes");
    const int lo = __builtin_amdgcn_update_dpp(x, x, 0x150 + src, 0xF, 0x3, false);
    return __int_as_float(__builtin_amdgcn_update_dpp(lo, x, 0x150 + 8 + src, 0xF, 0xC, false));
  }
}

struct SweepArgs {
  const float* ub;    // U block in LDS, [OB][OB]
  const float* pb;    // P block in LDS (drift only)
  const float* rinv;  // 1 / U_jj
  int sub, cb;
  float scale, inv_s, fzero, fmaxq;
  double dscale;
};

// one column of the sweep: j = 8 * OWN + S (compile-time)
template <bool DRIFT, int OWN, int S>
__device__ __forceinline__ void sweep_col(float (&w)[SweepLayout<DRIFT>::CPL],
                                          float (&ev)[SweepLayout<DRIFT>::CPL],
                                          float (&xv)[SweepLayout<DRIFT>::CPL],
                                          uint32_t (&qc)[SweepLayout<DRIFT>::CPL],
                                          const SweepArgs& a) {
  constexpr int LPR = SweepLayout<DRIFT>::LPR, CPL = SweepLayout<DRIFT>::CPL;
  constexpr int j = OWN * CPL + S;
  const float x = w[S];
  const float t = x * a.inv_s;
  float qf = __builtin_rintf(t);
  const bool tie = fabsf(t - floorf(t) - 0.5f) <= 1e-6f * (fabsf(t) + 1.f);
  if (tie && a.sub == OWN) qf = float(__builtin_rint(double(x) / a.dscale));
  const float q = fminf(fmaxf(qf + a.fzero, 0.f), a.fmaxq);
  const float wh = a.scale * (q - a.fzero);
  const float e = (x - wh) * a.rinv[j];
  if (a.sub == OWN) {
    ev[S] = e;
    qc[S] = uint32_t(q);
    if (DRIFT) xv[S] = x;
  }
  const float eb = row_bcast<LPR, OWN>(e);
#pragma unroll
  for (int h = 0; h < CPL / 4; ++h) {
    const float4 u = *reinterpret_cast<const float4*>(a.ub + j * OB + a.cb + 4 * h);
    w[4 * h + 0] = fmaf(-eb, u.x, w[4 * h + 0]);
    w[4 * h + 1] = fmaf(-eb, u.y, w[4 * h + 1]);
    w[4 * h + 2] = fmaf(-eb, u.z, w[4 * h + 2]);
    w[4 * h + 3] = fmaf(-eb, u.w, w[4 * h + 3]);
  }
  if (DRIFT) {  // + w_j P[j, its columns], w_j as it stood before quantisation
    const float xb = row_bcast<LPR, OWN>(x);
#pragma unroll
    for (int h = 0; h < CPL / 4; ++h) {
      const float4 pv = *reinterpret_cast<const float4*>(a.pb + j * OB + a.cb + 4 * h);
      w[4 * h + 0] = fmaf(xb, pv.x, w[4 * h + 0]);
      w[4 * h + 1] = fmaf(xb, pv.y, w[4 * h + 1]);
      w[4 * h + 2] = fmaf(xb, pv.z, w[4 * h + 2]);
      w[4 * h + 3] = fmaf(xb, pv.w, w[4 * h + 3]);
    }
  }
}

template <bool DRIFT, int OWN, int... S>
__device__ __forceinline__ void sweep_lane_cols(std::integer_sequence<int, S...>,
                                                float (&w)[SweepLayout<DRIFT>::CPL],
                                                float (&ev)[SweepLayout<DRIFT>::CPL],
                                                float (&xv)[SweepLayout<DRIFT>::CPL],
                                                uint32_t (&qc)[SweepLayout<DRIFT>::CPL],
                                                const SweepArgs& a) {
  (sweep_col<DRIFT, OWN, S>(w, ev, xv, qc, a), ...);
}

template <bool DRIFT, int... OWN>
__device__ __forceinline__ void sweep_all(std::integer_sequence<int, OWN...>,
                                          float (&w)[SweepLayout<DRIFT>::CPL],
                                          float (&ev)[SweepLayout<DRIFT>::CPL],
                                          float (&xv)[SweepLayout<DRIFT>::CPL],
                                          uint32_t (&qc)[SweepLayout<DRIFT>::CPL],
                                          const SweepArgs& a) {
  (sweep_lane_cols<DRIFT, OWN>(std::make_integer_sequence<int, SweepLayout<DRIFT>::CPL>{}, w, ev,
                               xv, qc, a),
   ...);
}

// (scale, zero) of a group from its range, the same float64 steps as the oracle's reading
__device__ __forceinline__ void grid_params(float xmin, float xmax, int bits, float& scale,
                                            float& fzero) {
  if (xmax == xmin) {
    xmin = -1.f;
    xmax = 1.f;
  }
  const double maxq = double((1 << bits) - 1);
  scale = float((double(xmax) - double(xmin)) / maxq);
  fzero = float(__builtin_rint(-double(xmin) / double(scale)));
}

// Group parameters of groups wider than one block: one wave per row reduces the row's current
// values over the group's columns [c0, c0 + g) (taken when the sweep reaches the group).
__global__ __launch_bounds__(256) void obs_group_params(const float* __restrict__ W,
                                                        int64_t d_out, int64_t ldw, int64_t c0,
                                                        int64_t g, int bits,
                                                        float* __restrict__ scales,
                                                        float* __restrict__ zeros, int64_t ldsz,
                                                        int64_t gi) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= d_out) return;  // uniform per wave
  const float* wr = W + row * ldw + c0;
  float xmin = 0.f, xmax = 0.f;
  for (int64_t c = int64_t(lane) * 4; c < g; c += 256) {
    const float4 v = *reinterpret_cast<const float4*>(wr + c);
    xmin = fminf(xmin, fminf(fminf(v.x, v.y), fminf(v.z, v.w)));
    xmax = fmaxf(xmax, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    xmin = fminf(xmin, __shfl_xor(xmin, o));
    xmax = fmaxf(xmax, __shfl_xor(xmax, o));
  }
  if (lane == 0) {
    float scale, fzero;
    grid_params(xmin, xmax, bits, scale, fzero);
    scales[row * ldsz + gi] = scale;
    zeros[row * ldsz + gi] = fzero;
  }
}

template <bool DRIFT>
__global__ __launch_bounds__(256) void obs_sweep(
    float* __restrict__ W, int64_t d_out, int64_t ldw, const float* __restrict__ U, int64_t ldu,
    const float* __restrict__ P, int64_t ldp, int64_t c0, int bits, uint8_t* __restrict__ codes,
    int64_t ldq, float* __restrict__ scales, float* __restrict__ zeros, int64_t ldsz, int64_t gi,
    int given, float* __restrict__ E, int64_t lde, float* __restrict__ Xq, int64_t ldxq,
    float* __restrict__ W_hat, int64_t ldwh) {
  __shared__ __attribute__((aligned(16))) float ub[OB * OB];  // U[c0 + j][c0 + k]
  __shared__ __attribute__((aligned(16))) float pb[DRIFT ? OB * OB : 4];  // P[c0 + j][c0 + k]
  __shared__ float rinv[OB];                                   // 1 / U_jj
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int LPR = SweepLayout<DRIFT>::LPR, CPL = SweepLayout<DRIFT>::CPL;
  constexpr int RPW = SweepLayout<DRIFT>::RPW, RPG = SweepLayout<DRIFT>::RPG;
  const int sub = lane & (LPR - 1), cb = sub * CPL;
  const int64_t row = int64_t(blockIdx.x) * RPG + wave * RPW + lane / LPR;
  const bool live = row < d_out;
  const int64_t rr = live ? row : d_out - 1;  // rows past the end recompute the last row

  for (int idx = tid; idx < OB * OB / 4; idx += 256) {
    const int j = idx / (OB / 4), k4 = (idx % (OB / 4)) * 4;
    *reinterpret_cast<float4*>(ub + j * OB + k4) =
        *reinterpret_cast<const float4*>(U + (c0 + j) * ldu + c0 + k4);
    if (DRIFT)
      *reinterpret_cast<float4*>(pb + j * OB + k4) =
          *reinterpret_cast<const float4*>(P + (c0 + j) * ldp + c0 + k4);
  }
  if (tid < OB) rinv[tid] = 1.f / U[(c0 + tid) * ldu + c0 + tid];
  float w[CPL];
#pragma unroll
  for (int h = 0; h < CPL / 4; ++h) {
    const float4 v = *reinterpret_cast<const float4*>(W + rr * ldw + c0 + cb + 4 * h);
    w[4 * h] = v.x, w[4 * h + 1] = v.y, w[4 * h + 2] = v.z, w[4 * h + 3] = v.w;
  }
  float scale, fzero;
  if (given) {  // a wider group: parameters taken at its first block by obs_group_params
    scale = scales[rr * ldsz + gi];
    fzero = zeros[rr * ldsz + gi];
  } else {  // group = block: parameters from the row's current 128 values
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
    grid_params(xmin, xmax, bits, scale, fzero);
  }
  __syncthreads();

  float ev[CPL], xv[CPL];
  uint32_t qc[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) ev[c] = 0.f, xv[c] = 0.f, qc[c] = 0u;
  const SweepArgs args{ub,          pb,    rinv, sub, cb, scale, 1.f / scale, fzero,
                       float((1 << bits) - 1), double(scale)};
  sweep_all<DRIFT>(std::make_integer_sequence<int, LPR>{}, w, ev, xv, qc, args);

  if (!live) return;
  if (sub == 0 && !given) {
    scales[row * ldsz + gi] = scale;
    zeros[row * ldsz + gi] = fzero;
  }
  float wh[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) wh[c] = scale * (float(qc[c]) - fzero);
#pragma unroll
  for (int h = 0; h < CPL / 4; ++h) {
    const float4 hv = make_float4(wh[4 * h], wh[4 * h + 1], wh[4 * h + 2], wh[4 * h + 3]);
    *reinterpret_cast<float4*>(W + row * ldw + c0 + cb + 4 * h) = hv;
    if (W_hat) *reinterpret_cast<float4*>(W_hat + row * ldwh + c0 + cb + 4 * h) = hv;
    *reinterpret_cast<float4*>(E + row * lde + cb + 4 * h) =
        make_float4(ev[4 * h], ev[4 * h + 1], ev[4 * h + 2], ev[4 * h + 3]);
    if (DRIFT)
      *reinterpret_cast<float4*>(Xq + row * ldxq + cb + 4 * h) =
          make_float4(xv[4 * h], xv[4 * h + 1], xv[4 * h + 2], xv[4 * h + 3]);
    reinterpret_cast<uint32_t*>(codes + row * ldq + c0 + cb)[h] =
        qc[4 * h] | (qc[4 * h + 1] << 8) | (qc[4 * h + 2] << 16) | (qc[4 * h + 3] << 24);
  }
}

// Blocks per lazy group for a quantisation group of `group` columns: a group's parameters need
// its columns current when the sweep reaches it, which holds when it lies inside one lazy group
// or starts one. 0 when the group is not supported.
int lazy_blocks(int64_t d_in, int group) {
  if (group < OB || group % OB != 0 || d_in % group != 0) return 0;
  const int m = group / OB;
  if (GRP % m == 0 || m % GRP == 0 || group == d_in) return GRP;
  for (int k = GRP - 1; k > 1; --k)
    if (m % k == 0) return k;
  return 1;
}

}  // namespace

int obs_group_ok(int64_t d_in, int group) { return lazy_blocks(d_in, group); }

size_t obs_ws_bytes(int64_t d_out, int64_t d_in, bool drift) {
  if (d_out <= 0 || d_in <= 0) return 0;
  const size_t per = align256(size_t(d_out) * GRP * OB * sizeof(float)) +
                     2 * align256(size_t(d_in) * size_t(d_in) * sizeof(uint16_t));
  return (drift ? 2 : 1) * per + 256;
}

int obs_launch(float* W, int64_t d_out, int64_t d_in, int64_t ldw, const float* U, int64_t ldu,
               int bits, int group, const float* P, int64_t ldp, uint8_t* codes, float* scales,
               float* zeros, float* err, float* W_hat, void* ws, hipStream_t s) {
  const bool drift = P != nullptr;
  const int64_t nblk = d_in / OB, ldsz = d_in / group;
  const int lz = lazy_blocks(d_in, group);
  KQ_REQUIRE(lz > 0, KRONQ_ERR_UNSUPPORTED, "group %d not supported for d_in %lld", group,
             (long long)d_in);
  const unsigned grid = unsigned(cdiv(d_out, drift ? SweepLayout<true>::RPG
                                                   : SweepLayout<false>::RPG));
  Carver cv(ws);
  float* Ews = cv.take<float>(size_t(d_out) * GRP * OB);
  uint16_t* Uth = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  uint16_t* Utl = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  float* Xws = drift ? cv.take<float>(size_t(d_out) * GRP * OB) : nullptr;
  uint16_t* Pth = drift ? cv.take<uint16_t>(size_t(d_in) * size_t(d_in)) : nullptr;
  uint16_t* Ptl = drift ? cv.take<uint16_t>(size_t(d_in) * size_t(d_in)) : nullptr;
  // U^T (and -P^T) split once into bf16 high and low parts: the B operands of the trailing
  // updates
  KQ_TRY(split_transpose_launch(U, ldu, d_in, Uth, Utl, d_in, s));
  if (drift) KQ_TRY(split_transpose_launch(P, ldp, d_in, Pth, Ptl, d_in, s, true));
  const int64_t ldx = GRP * OB;
  for (int64_t g0 = 0; g0 < nblk; g0 += lz) {
    const int64_t gend = g0 + lz < nblk ? g0 + lz : nblk;
    // errors of this lazy group's blocks: the caller's err (ld d_in) or the workspace
    // (ld GRP * OB); pre-quantisation values (drift) always in the workspace
    float* Eg = err ? err + g0 * OB : Ews;
    const int64_t lde = err ? d_in : GRP * OB;
    for (int64_t b = g0; b < gend; ++b) {
      const int64_t c0 = b * OB;
      float* Eb = Eg + (b - g0) * OB;
      float* Xb = drift ? Xws + (b - g0) * OB : nullptr;
      const int64_t gi = c0 / group;
      const int given = group > OB;
      if (given && c0 % group == 0)
        KQ_TRY(launch("obs_group_params", obs_group_params, dim3(unsigned(cdiv(d_out, 4))),
                      dim3(256), 0, s, static_cast<const float*>(W), d_out, ldw, c0,
                      int64_t(group), bits, scales, zeros, ldsz, gi));
      if (drift)
        KQ_TRY(launch("obs_sweep", obs_sweep<true>, dim3(grid), dim3(256), 0, s, W, d_out, ldw, U,
                      ldu, P, ldp, c0, bits, codes, d_in, scales, zeros, ldsz, gi, given, Eb, lde,
                      Xb, ldx, W_hat, d_in));
      else
        KQ_TRY(launch("obs_sweep", obs_sweep<false>, dim3(grid), dim3(256), 0, s, W, d_out, ldw,
                      U, ldu, P, ldp, c0, bits, codes, d_in, scales, zeros, ldsz, gi, given, Eb,
                      lde, Xb, ldx, W_hat, d_in));
      const int64_t near = (gend - b - 1) * OB;  // rest of the lazy group
      if (near > 0) {
        // W[:, c0+OB : gend*OB] -= E_b U[c0 : c0+OB, c0+OB : gend*OB] (- X_b P[...])
        Bf16x3Pair pu{Eb, lde, Uth + (c0 + OB) * d_in + c0, Utl + (c0 + OB) * d_in + c0, d_in,
                      OB};
        Bf16x3Pair pp;
        if (drift)
          pp = Bf16x3Pair{Xb, ldx, Pth + (c0 + OB) * d_in + c0, Ptl + (c0 + OB) * d_in + c0,
                          d_in, OB};
        KQ_TRY(gemm_bf16x3_sub(d_out, near, pu, pp, W + c0 + OB, ldw, s, "obs_trailing_update"));
      }
    }
    const int64_t rem = d_in - gend * OB;  // beyond the lazy group
    if (rem > 0) {
      // W[:, gend*OB :] -= E_group U[g0*OB : gend*OB, gend*OB :] (- X_group P[...])
      const int64_t K = (gend - g0) * OB, off = gend * OB * d_in + g0 * OB;
      Bf16x3Pair pu{Eg, lde, Uth + off, Utl + off, d_in, K};
      Bf16x3Pair pp;
      if (drift) pp = Bf16x3Pair{Xws, ldx, Pth + off, Ptl + off, d_in, K};
      KQ_TRY(gemm_bf16x3_sub(d_out, rem, pu, pp, W + gend * OB, ldw, s, "obs_trailing_update"));
    }
  }
  return KRONQ_OK;
}

}  // namespace kq
