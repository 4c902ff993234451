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

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// round-to-nearest-even fp32 -> bf16 bits (finite inputs)
__device__ __forceinline__ uint32_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

constexpr int OB = 128;          // block (and the smallest group)
constexpr int LZMAX = 4;         // blocks per lazy group of the P = 0 sweep (at most)
// Lanes per row of the sweep kernel, a template parameter: 8 (16 columns per lane, 8 rows per
// wave) or 16 (8 columns per lane, 4 rows per wave). 8 lanes halve the instructions per row,
// which matters when the rows are many and the sweep is throughput-bound (d_out = 28672, or on
// part of the chip beside the H_G covariance); 16 lanes give twice the waves for a small d_out,
// whose sweep is latency-bound on the whole chip (d_out = 4096 alone: 20.6 against 26.2 us per
// block). The drift correction uses 16: its second broadcast and P block would not fit the
// registers of 16 columns.
template <int L>
struct SweepLayout {
  static constexpr int LPR = L;          // lanes per row
  static constexpr int CPL = OB / L;     // columns per lane
  static constexpr int RPW = 64 / L;     // rows per wave
  static constexpr int RPG = 4 * RPW;    // rows per workgroup (4 waves)
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

// an empty asm statement that reads and writes every element: its value must exist here
template <int N>
__device__ __forceinline__ void pin_regs(float (&w)[N]) {
  static_assert(N % 4 == 0, "groups of four");
#pragma unroll
  for (int h = 0; h < N / 4; ++h)
    asm volatile("" : "+v"(w[4 * h]), "+v"(w[4 * h + 1]), "+v"(w[4 * h + 2]), "+v"(w[4 * h + 3]));
}

struct SweepArgs {
  const float* ub;    // U block in LDS, [OB][OB]
  const float* pb;    // P block in LDS (drift only)
  const float* rinv;  // 1 / U_jj
  int sub, cb;
  float scale, inv_s, fzero, fmaxq;
  double dscale;
};

// one column of the sweep: j = CPL * OWN + S (compile-time). uc / rc hold U[j, this lane's
// columns] and 1 / U_jj, read from LDS during the previous column; this column issues the reads
// for column j + 1 first, so that their latency is hidden behind its own work.
template <bool DRIFT, int L, int OWN, int S>
__device__ __forceinline__ void sweep_col(float (&w)[SweepLayout<L>::CPL],
                                          float (&ev)[SweepLayout<L>::CPL],
                                          float (&xv)[SweepLayout<L>::CPL],
                                          uint32_t (&qc)[SweepLayout<L>::CPL],
                                          float (&uc)[SweepLayout<L>::CPL], float& rc,
                                          const SweepArgs& a) {
  constexpr int LPR = SweepLayout<L>::LPR, CPL = SweepLayout<L>::CPL;
  constexpr int j = OWN * CPL + S;
  float un[CPL];
  float rn = 0.f;
  if constexpr (j + 1 < OB) {
#pragma unroll
    for (int h = 0; h < CPL / 4; ++h) {
      const float4 u = *reinterpret_cast<const float4*>(a.ub + (j + 1) * OB + a.cb + 4 * h);
      un[4 * h] = u.x, un[4 * h + 1] = u.y, un[4 * h + 2] = u.z, un[4 * h + 3] = u.w;
    }
    rn = a.rinv[j + 1];
  }
  __builtin_amdgcn_sched_barrier(0);  // the reads go out before this column's work
  const float x = w[S];
  const float t = x * a.inv_s;
  float qf = __builtin_rintf(t);
  const bool tie = fabsf(t - floorf(t) - 0.5f) <= 1e-6f * (fabsf(t) + 1.f);
  if (tie && a.sub == OWN) qf = float(__builtin_rint(double(x) / a.dscale));
  const float q = fminf(fmaxf(qf + a.fzero, 0.f), a.fmaxq);
  const float wh = a.scale * (q - a.fzero);
  const float e = (x - wh) * rc;
  if (a.sub == OWN) {
    ev[S] = e;
    qc[S] = uint32_t(q);
    if (DRIFT) xv[S] = x;
  }
  const float eb = row_bcast<LPR, OWN>(e);
  // the next column's update first: it is the one the next quantisation waits for
  constexpr int nxt = (S + 1) % CPL;
  w[nxt] = fmaf(-eb, uc[nxt], w[nxt]);
#pragma unroll
  for (int c = 0; c < CPL; ++c)
    if (c != nxt) w[c] = fmaf(-eb, uc[c], w[c]);
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
  // the column's updates are applied here, as soon as e_j exists: left to itself the compiler
  // sinks each column's FMAs to just before that column is quantised, which turns them into
  // one long chain of dependent FMAs on the sweep's critical path (and keeps every e_j and U
  // value live in registers). An empty asm that reads and writes every w pins them here.
  pin_regs(w);
#pragma unroll
  for (int c = 0; c < CPL; ++c) uc[c] = un[c];
  rc = rn;
}

template <bool DRIFT, int L, int OWN, int... S>
__device__ __forceinline__ void sweep_lane_cols(std::integer_sequence<int, S...>,
                                                float (&w)[SweepLayout<L>::CPL],
                                                float (&ev)[SweepLayout<L>::CPL],
                                                float (&xv)[SweepLayout<L>::CPL],
                                                uint32_t (&qc)[SweepLayout<L>::CPL],
                                                float (&uc)[SweepLayout<L>::CPL], float& rc,
                                                const SweepArgs& a) {
  (sweep_col<DRIFT, L, OWN, S>(w, ev, xv, qc, uc, rc, a), ...);
}

template <bool DRIFT, int L, int... OWN>
__device__ __forceinline__ void sweep_all(std::integer_sequence<int, OWN...>,
                                          float (&w)[SweepLayout<L>::CPL],
                                          float (&ev)[SweepLayout<L>::CPL],
                                          float (&xv)[SweepLayout<L>::CPL],
                                          uint32_t (&qc)[SweepLayout<L>::CPL],
                                          const SweepArgs& a) {
  float uc[SweepLayout<L>::CPL];
  constexpr int CPL = SweepLayout<L>::CPL;
#pragma unroll
  for (int h = 0; h < CPL / 4; ++h) {  // U row 0
    const float4 u = *reinterpret_cast<const float4*>(a.ub + a.cb + 4 * h);
    uc[4 * h] = u.x, uc[4 * h + 1] = u.y, uc[4 * h + 2] = u.z, uc[4 * h + 3] = u.w;
  }
  float rc = a.rinv[0];
  (sweep_lane_cols<DRIFT, L, OWN>(std::make_integer_sequence<int, CPL>{}, w, ev, xv, qc, uc,
                                  rc, a),
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

// Pending updates of this block (the P = 0 sweep): the workgroup's rows of
// W[:, c0 : c0 + OB] still owe sum_k E[row, k] U[kp0 + k, c0 + n] over the kpend columns of the
// lazy group swept before this block. One 32 x 32 MFMA block per wave (its 32 of the block's
// 128 columns, rows row0 .. row0 + 31), K in steps of 16, on the bf16 matrix cores with the
// three-term split: the earlier blocks' errors (Efh, Efl) and U^T (Ufh, Ufl) come split and in
// MFMA-fragment order (split_frag_index), so that each fragment load of a wave is one contiguous
// kilobyte (row-major operands cost 32 cache lines per load, which made this step take as long
// as the column sweep itself). K runs in 64-wide steps whose 16 fragment loads are requested one
// step ahead of the step's 12 MFMAs, and the three products accumulate separately (three
// independent MFMA chains, summed at the end). The result lands in dl[row - row0][column].
constexpr int EKS = LZMAX * OB / 16;  // 16-k units per 32-row group of the errors
__device__ __forceinline__ void pending_update(const uint16_t* __restrict__ Efh,
                                               const uint16_t* __restrict__ Efl,
                                               const uint16_t* __restrict__ Ufh,
                                               const uint16_t* __restrict__ Ufl, int64_t d_in,
                                               int64_t kp0, int kpend, int64_t c0,
                                               int64_t row0, int64_t d_out, int wave, int lane,
                                               float (*dl)[OB + 4]) {
  constexpr int KS = 64;  // k per step
  const int l32 = lane & 31, lhi = lane >> 5;
  const int64_t ra = row0 + l32 < d_out ? row0 + l32 : d_out - 1;  // rows past the end: unused
  const int64_t eo = split_frag_index(ra, 8 * lhi, EKS);
  const uint16_t* eh = Efh + eo;
  const uint16_t* el = Efl + eo;
  const int64_t uo = split_frag_index(c0 + wave * 32 + l32, kp0 + 8 * lhi, d_in / 16);
  const uint16_t* bh = Ufh + uo;
  const uint16_t* bl = Ufl + uo;
  f32x16_t hh = {}, lh = {}, hl = {};
  bf16x8_t f0[4][KS / 16], f1[4][KS / 16];  // [eh, el, uh, ul][k step of 16]
  auto load = [&](bf16x8_t (&f)[4][KS / 16], int k0) {
#pragma unroll
    for (int ks = 0; ks < KS / 16; ++ks) {
      const int kk = (k0 + 16 * ks) * 32;  // next 16-k unit: 512 elements on
      f[0][ks] = *reinterpret_cast<const bf16x8_t*>(eh + kk);
      f[1][ks] = *reinterpret_cast<const bf16x8_t*>(el + kk);
      f[2][ks] = *reinterpret_cast<const bf16x8_t*>(bh + kk);
      f[3][ks] = *reinterpret_cast<const bf16x8_t*>(bl + kk);
    }
  };
  auto mfmas = [&](const bf16x8_t (&f)[4][KS / 16]) {
#pragma unroll
    for (int ks = 0; ks < KS / 16; ++ks) {
      lh = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[1][ks], f[2][ks], lh, 0, 0, 0);
      hl = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[0][ks], f[3][ks], hl, 0, 0, 0);
      hh = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[0][ks], f[2][ks], hh, 0, 0, 0);
    }
  };
  // kpend is a multiple of 128: steps in pairs, the loads of each step one step ahead. The
  // load after the last pair is issued too (it re-reads the last step, in bounds): a skipped
  // load would make the wait before the second half's MFMAs a full one on every pair.
  // (The scheduling barriers keep each step's loads ahead of the other step's MFMAs; left to
  // itself the compiler interleaves them and each MFMA waits for a load issued just before.)
  load(f0, 0);
  for (int k0 = 0; k0 < kpend; k0 += 2 * KS) {
    load(f1, k0 + KS);
    __builtin_amdgcn_sched_barrier(0);
    mfmas(f0);
    __builtin_amdgcn_sched_barrier(0);
    load(f0, k0 + 2 * KS < kpend ? k0 + 2 * KS : kpend - KS);
    __builtin_amdgcn_sched_barrier(0);
    mfmas(f1);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r)
    dl[8 * (r >> 2) + 4 * lhi + (r & 3)][wave * 32 + l32] = (lh[r] + hl[r]) + hh[r];
}

template <bool DRIFT, int L>
__global__ __launch_bounds__(256) void obs_sweep(
    float* __restrict__ W, int64_t d_out, int64_t ldw, const float* __restrict__ U, int64_t ldu,
    const float* __restrict__ P, int64_t ldp, int64_t c0, int bits, uint8_t* __restrict__ codes,
    int64_t ldq, float* __restrict__ scales, float* __restrict__ zeros, int64_t ldsz, int64_t gi,
    int given, float* __restrict__ E, int64_t lde, float* __restrict__ Xq, int64_t ldxq,
    float* __restrict__ W_hat, int64_t ldwh, uint16_t* __restrict__ Eh,
    uint16_t* __restrict__ El, int64_t ldes, uint16_t* __restrict__ Efh,
    uint16_t* __restrict__ Efl, const uint16_t* __restrict__ Ufh,
    const uint16_t* __restrict__ Ufl, int64_t d_in, int64_t kp0, int kpend) {
  __shared__ __attribute__((aligned(16))) float ub[OB * OB];  // U[c0 + j][c0 + k]
  __shared__ __attribute__((aligned(16))) float pb[DRIFT ? OB * OB : 4];  // P[c0 + j][c0 + k]
  __shared__ float rinv[OB];                                   // 1 / U_jj
  constexpr int LPR = SweepLayout<L>::LPR, CPL = SweepLayout<L>::CPL;
  constexpr int RPW = SweepLayout<L>::RPW, RPG = SweepLayout<L>::RPG;
  // pending update: 32 rows (one MFMA block; with 16 rows per workgroup the second half is
  // computed and left unused)
  __shared__ __attribute__((aligned(16))) float dl[DRIFT ? 1 : 32][OB + 4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane & (LPR - 1), cb = sub * CPL;
  const int64_t row = int64_t(blockIdx.x) * RPG + wave * RPW + lane / LPR;
  const bool live = row < d_out;
  const int64_t rr = live ? row : d_out - 1;  // rows past the end recompute the last row

  // the U (and P) block: every load requested before the first store (a load-store pair per
  // iteration would wait out one memory latency per iteration)
  {
    constexpr int NV = OB * OB / 4 / 256;
    float4 uv[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = tid + 256 * i, j = idx / (OB / 4), k4 = (idx % (OB / 4)) * 4;
      uv[i] = *reinterpret_cast<const float4*>(U + (c0 + j) * ldu + c0 + k4);
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) reinterpret_cast<float4*>(ub)[tid + 256 * i] = uv[i];
    if (DRIFT) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int idx = tid + 256 * i, j = idx / (OB / 4), k4 = (idx % (OB / 4)) * 4;
        uv[i] = *reinterpret_cast<const float4*>(P + (c0 + j) * ldp + c0 + k4);
      }
#pragma unroll
      for (int i = 0; i < NV; ++i) reinterpret_cast<float4*>(pb)[tid + 256 * i] = uv[i];
    }
  }
  if (tid < OB) rinv[tid] = 1.f / U[(c0 + tid) * ldu + c0 + tid];
  float w[CPL];
#pragma unroll
  for (int h = 0; h < CPL / 4; ++h) {
    const float4 v = *reinterpret_cast<const float4*>(W + rr * ldw + c0 + cb + 4 * h);
    w[4 * h] = v.x, w[4 * h + 1] = v.y, w[4 * h + 2] = v.z, w[4 * h + 3] = v.w;
  }
  if constexpr (!DRIFT) {
    if (kpend > 0) {  // uniform over the launch
      pending_update(Efh, Efl, Ufh, Ufl, d_in, kp0, kpend, c0, int64_t(blockIdx.x) * RPG, d_out,
                     wave, lane, dl);
      __syncthreads();
      const int rl = wave * RPW + lane / LPR;
#pragma unroll
      for (int h = 0; h < CPL / 4; ++h) {
        const float4 v = *reinterpret_cast<const float4*>(&dl[rl][cb + 4 * h]);
        w[4 * h] -= v.x, w[4 * h + 1] -= v.y, w[4 * h + 2] -= v.z, w[4 * h + 3] -= v.w;
      }
    }
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
  sweep_all<DRIFT, L>(std::make_integer_sequence<int, LPR>{}, w, ev, xv, qc, args);

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
    if (E)
      *reinterpret_cast<float4*>(E + row * lde + cb + 4 * h) =
          make_float4(ev[4 * h], ev[4 * h + 1], ev[4 * h + 2], ev[4 * h + 3]);
    if (!DRIFT) {  // the errors split into bf16 high and low parts for the products after it
      uint32_t hi[2], lo[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const uint32_t h0 = bf16_rne(ev[4 * h + 2 * e]), h1 = bf16_rne(ev[4 * h + 2 * e + 1]);
        const uint32_t l0 = bf16_rne(ev[4 * h + 2 * e] - __uint_as_float(h0 << 16));
        const uint32_t l1 = bf16_rne(ev[4 * h + 2 * e + 1] - __uint_as_float(h1 << 16));
        hi[e] = h0 | (h1 << 16);
        lo[e] = l0 | (l1 << 16);
      }
      *reinterpret_cast<uint2*>(Eh + row * ldes + cb + 4 * h) = make_uint2(hi[0], hi[1]);
      *reinterpret_cast<uint2*>(El + row * ldes + cb + 4 * h) = make_uint2(lo[0], lo[1]);
      // and in fragment order for the in-kernel updates of the later blocks of the lazy group
      // (column kpend + cb + 4 h of the group; four bf16 never straddle an 8-k fragment)
      const int64_t f = split_frag_index(row, kpend + cb + 4 * h, EKS);
      *reinterpret_cast<uint2*>(Efh + f) = make_uint2(hi[0], hi[1]);
      *reinterpret_cast<uint2*>(Efl + f) = make_uint2(lo[0], lo[1]);
    }
    if (DRIFT)
      *reinterpret_cast<float4*>(Xq + row * ldxq + cb + 4 * h) =
          make_float4(xv[4 * h], xv[4 * h + 1], xv[4 * h + 2], xv[4 * h + 3]);
    reinterpret_cast<uint32_t*>(codes + row * ldq + c0 + cb)[h] =
        qc[4 * h] | (qc[4 * h + 1] << 8) | (qc[4 * h + 2] << 16) | (qc[4 * h + 3] << 24);
  }
}

// Blocks per lazy group for a quantisation group of `group` columns: a group's parameters need
// its columns current when the sweep reaches it, which holds when it lies inside one lazy group
// or starts one. 0 when the group is not supported. (Drift path: the near updates are applied
// after every block, so the whole lazy group is current.)
int lazy_blocks(int64_t d_in, int group) {
  if (group < OB || group % OB != 0 || d_in % group != 0) return 0;
  const int m = group / OB;
  if (GRP % m == 0 || m % GRP == 0 || group == d_in) return GRP;
  for (int k = GRP - 1; k > 1; --k)
    if (m % k == 0) return k;
  return 1;
}

// Blocks per lazy group of the P = 0 sweep, whose pending updates reach a block only when the
// sweep gets there: a quantisation group's columns are all current at its first block only if
// that block starts a lazy group (then every earlier update has been applied to everything after
// it). So the lazy group divides the quantisation group (up to LZMAX blocks); a group of one
// block, or the whole row (parameters from the initial row), allows LZMAX.
int lazy_blocks_pending(int64_t d_in, int group) {
  if (group < OB || group % OB != 0 || d_in % group != 0) return 0;
  const int m = group / OB;
  if (m == 1 || group == d_in) return LZMAX;
  for (int k = m < LZMAX ? m : LZMAX; k > 1; --k)
    if (m % k == 0) return k;
  return 1;
}

}  // namespace

int obs_group_ok(int64_t d_in, int group) { return lazy_blocks(d_in, group); }

size_t obs_ws_bytes(int64_t d_out, int64_t d_in, bool drift) {
  if (d_out <= 0 || d_in <= 0) return 0;
  const size_t split_u = 2 * align256(size_t(d_in) * size_t(d_in) * sizeof(uint16_t));
  if (!drift)  // split errors of a lazy group and split U^T, row-major and in fragment order
    return 2 * align256(size_t(d_out) * LZMAX * OB * sizeof(uint16_t)) +
           2 * align256(size_t(cdiv(d_out, 32) * 32) * LZMAX * OB * sizeof(uint16_t)) +
           2 * split_u + 256;
  // errors and pre-quantisation values of a lazy group, split U^T and -P^T
  return 2 * (align256(size_t(d_out) * GRP * OB * sizeof(float)) + split_u) + 256;
}

namespace {

// P = 0: one sweep launch per block, which first applies the updates the block still owes to
// the earlier blocks of its lazy group (pending_update), then one trailing product per lazy
// group for everything after it.
int obs_launch_pending(float* W, int64_t d_out, int64_t d_in, int64_t ldw, const float* U,
                       int64_t ldu, int bits, int group, uint8_t* codes, float* scales,
                       float* zeros, float* err, float* W_hat, void* ws, hipStream_t s) {
  const int64_t nblk = d_in / OB, ldsz = d_in / group;
  const int lz = lazy_blocks_pending(d_in, group);
  KQ_REQUIRE(lz > 0, KRONQ_ERR_UNSUPPORTED, "group %d not supported for d_in %lld", group,
             (long long)d_in);
  // 16 lanes per row only for a small d_out: beside the H_G covariance the sweep has part of
  // the chip, where the 16-lane layout's twice as many workgroups (one per CU) take two rounds
  // (8B q_proj layer: 11.31-11.39 ms per layer with 8 lanes, 11.46-11.48 with 16)
  const bool lanes16 = d_out <= 2048;
  const unsigned grid =
      unsigned(cdiv(d_out, lanes16 ? SweepLayout<16>::RPG : SweepLayout<8>::RPG));
  Carver cv(ws);
  // the lazy group's errors, split into bf16 high and low parts [row][LZMAX * OB]
  const int64_t ldes = LZMAX * OB;
  uint16_t* Eh = cv.take<uint16_t>(size_t(d_out) * ldes);
  uint16_t* El = cv.take<uint16_t>(size_t(d_out) * ldes);
  uint16_t* Uth = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  uint16_t* Utl = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  // the same two, in MFMA-fragment order, for the sweep's in-kernel updates
  uint16_t* Efh = cv.take<uint16_t>(size_t(cdiv(d_out, 32) * 32) * ldes);
  uint16_t* Efl = cv.take<uint16_t>(size_t(cdiv(d_out, 32) * 32) * ldes);
  uint16_t* Ufh = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  uint16_t* Ufl = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  KQ_TRY(split_transpose_launch(U, ldu, d_in, Uth, Utl, d_in, s, false, Ufh, Ufl));
  for (int64_t g0 = 0; g0 < nblk; g0 += lz) {
    const int64_t gend = g0 + lz < nblk ? g0 + lz : nblk;
    for (int64_t b = g0; b < gend; ++b) {
      const int64_t c0 = b * OB, gi = c0 / group, eo = (b - g0) * OB;
      const int given = group > OB;
      if (given && c0 % group == 0)
        KQ_TRY(launch("obs_group_params", obs_group_params, dim3(unsigned(cdiv(d_out, 4))),
                      dim3(256), 0, s, static_cast<const float*>(W), d_out, ldw, c0,
                      int64_t(group), bits, scales, zeros, ldsz, gi));
      KQ_TRY(launch("obs_sweep", lanes16 ? obs_sweep<false, 16> : obs_sweep<false, 8>,
                    dim3(grid), dim3(256), 0, s, W, d_out, ldw, U, ldu,
                    static_cast<const float*>(nullptr), int64_t(0), c0, bits, codes, d_in,
                    scales, zeros, ldsz, gi, given, err ? err + c0 : static_cast<float*>(nullptr),
                    d_in, static_cast<float*>(nullptr), int64_t(0), W_hat, d_in, Eh + eo, El + eo,
                    ldes, Efh, Efl, static_cast<const uint16_t*>(Ufh),
                    static_cast<const uint16_t*>(Ufl), d_in, g0 * OB, int(eo)));
    }
    const int64_t rem = d_in - gend * OB;  // beyond the lazy group
    if (rem > 0) {
      // W[:, gend*OB :] -= E_group U[g0*OB : gend*OB, gend*OB :]
      const int64_t K = (gend - g0) * OB, off = gend * OB * d_in + g0 * OB;
      KQ_TRY(gemm_bf16x3_presplit_sub(d_out, rem, K, Eh, El, ldes, Uth + off, Utl + off, d_in,
                                      W + gend * OB, ldw, s, "obs_trailing_update"));
    }
  }
  return KRONQ_OK;
}

}  // namespace

int obs_launch(float* W, int64_t d_out, int64_t d_in, int64_t ldw, const float* U, int64_t ldu,
               int bits, int group, const float* P, int64_t ldp, uint8_t* codes, float* scales,
               float* zeros, float* err, float* W_hat, void* ws, hipStream_t s) {
  if (P == nullptr)
    return obs_launch_pending(W, d_out, d_in, ldw, U, ldu, bits, group, codes, scales, zeros,
                              err, W_hat, ws, s);
  // the drift correction: two-level lazy updates, near ones after every block
  const int64_t nblk = d_in / OB, ldsz = d_in / group;
  const int lz = lazy_blocks(d_in, group);
  KQ_REQUIRE(lz > 0, KRONQ_ERR_UNSUPPORTED, "group %d not supported for d_in %lld", group,
             (long long)d_in);
  const unsigned grid = unsigned(cdiv(d_out, SweepLayout<16>::RPG));
  Carver cv(ws);
  float* Ews = cv.take<float>(size_t(d_out) * GRP * OB);
  uint16_t* Uth = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  uint16_t* Utl = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  float* Xws = cv.take<float>(size_t(d_out) * GRP * OB);
  uint16_t* Pth = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  uint16_t* Ptl = cv.take<uint16_t>(size_t(d_in) * size_t(d_in));
  // U^T and -P^T split once into bf16 high and low parts: the B operands of the trailing
  // updates
  KQ_TRY(split_transpose_launch(U, ldu, d_in, Uth, Utl, d_in, s));
  KQ_TRY(split_transpose_launch(P, ldp, d_in, Pth, Ptl, d_in, s, true));
  const int64_t ldx = GRP * OB;
  for (int64_t g0 = 0; g0 < nblk; g0 += lz) {
    const int64_t gend = g0 + lz < nblk ? g0 + lz : nblk;
    float* Eg = err ? err + g0 * OB : Ews;
    const int64_t lde = err ? d_in : GRP * OB;
    for (int64_t b = g0; b < gend; ++b) {
      const int64_t c0 = b * OB;
      float* Eb = Eg + (b - g0) * OB;
      float* Xb = Xws + (b - g0) * OB;
      const int64_t gi = c0 / group;
      const int given = group > OB;
      if (given && c0 % group == 0)
        KQ_TRY(launch("obs_group_params", obs_group_params, dim3(unsigned(cdiv(d_out, 4))),
                      dim3(256), 0, s, static_cast<const float*>(W), d_out, ldw, c0,
                      int64_t(group), bits, scales, zeros, ldsz, gi));
      KQ_TRY(launch("obs_sweep", obs_sweep<true, 16>, dim3(grid), dim3(256), 0, s, W, d_out, ldw, U,
                    ldu, P, ldp, c0, bits, codes, d_in, scales, zeros, ldsz, gi, given, Eb, lde,
                    Xb, ldx, W_hat, d_in, static_cast<uint16_t*>(nullptr),
                    static_cast<uint16_t*>(nullptr), int64_t(0), static_cast<uint16_t*>(nullptr),
                    static_cast<uint16_t*>(nullptr), static_cast<const uint16_t*>(nullptr),
                    static_cast<const uint16_t*>(nullptr), d_in, int64_t(0), 0));
      const int64_t near = (gend - b - 1) * OB;  // rest of the lazy group
      if (near > 0) {
        // W[:, c0+OB : gend*OB] -= E_b U[c0 : c0+OB, c0+OB : gend*OB] - X_b P[...]
        Bf16x3Pair pu{Eb, lde, Uth + (c0 + OB) * d_in + c0, Utl + (c0 + OB) * d_in + c0, d_in,
                      OB};
        Bf16x3Pair pp{Xb, ldx, Pth + (c0 + OB) * d_in + c0, Ptl + (c0 + OB) * d_in + c0, d_in,
                      OB};
        KQ_TRY(gemm_bf16x3_sub(d_out, near, pu, pp, W + c0 + OB, ldw, s, "obs_trailing_update"));
      }
    }
    const int64_t rem = d_in - gend * OB;  // beyond the lazy group
    if (rem > 0) {
      const int64_t K = (gend - g0) * OB, off = gend * OB * d_in + g0 * OB;
      Bf16x3Pair pu{Eg, lde, Uth + off, Utl + off, d_in, K};
      Bf16x3Pair pp{Xws, ldx, Pth + off, Ptl + off, d_in, K};
      KQ_TRY(gemm_bf16x3_sub(d_out, rem, pu, pp, W + gend * OB, ldw, s, "obs_trailing_update"));
    }
  }
  return KRONQ_OK;
}

}  // namespace kq
