// Covariance accumulation H <- beta H + alpha A^T A (Sec. 4.1 eq. kfac; Alg. 1 first line), and
// the drift statistic C <- beta C + alpha A^T B (Alg. 1 first line, dX X^T in token-major form)
// with the same kernels over all tiles instead of the upper triangle ("cross" below).
//
// bf16 path: a syrk on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16). bf16 x bf16 products
// are exact in fp32 and accumulate in fp32.
//   * Work split: the token dimension is cut into S slices (split-K). S is chosen so that the
//     tiles x slices workgroups fill whole rounds of the CUs, in multiples of 8 that keep each
//     XCD on its own slices (see cov_plan).
//   * Each workgroup owns one 256 x 256 tile (I <= J; any I, J for cross) of H for its slice:
//     4 waves, each a 128 x 128 sub-tile = 4 x 4 MFMA blocks of 32 x 32, 256 fp32
//     accumulators per lane.
//   * Interior tiles (syrk_bf16_dma below) stream 32-token stages straight from HBM into a
//     ring of LDS buffers and transpose on the LDS read. Tiles of a ragged last channel block
//     and a ragged token tail (< 32 tokens) go through syrk_bf16_partial, which stages 64
//     tokens through registers: 8 x 8 bf16 blocks are loaded, transposed with v_perm and
//     written token-contiguous to LDS so that an MFMA operand is one 16-byte read.
//   * Partial tiles go to the workspace in MFMA-fragment order; a reduction kernel sums the
//     slices, applies alpha/beta and writes both triangles (the mirror through an LDS
//     transpose), so H is exactly symmetric; for cross every tile is written as it is.
// fp32 path (small fp32 inputs): a plain LDS-tiled fp32 FMA kernel over the full matrix.
#include <algorithm>
#include <cmath>
#include <type_traits>
#include <utility>

#include "kq_common.hpp"

namespace kq {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int TT = 256;       // output tile edge
constexpr int KC = 64;        // tokens per stage
constexpr int LROW = 36;      // LDS row stride in dwords (64 bf16 + 8 pad)
constexpr int OPER = TT * LROW;  // dwords per operand buffer

__device__ __forceinline__ u32x4_t load_row8(const uint16_t* __restrict__ A, int64_t lda,
                                             int64_t t, int64_t t_end, int64_t col, int64_t d) {
  u32x4_t v = {0u, 0u, 0u, 0u};
  if (t >= t_end) return v;
  const uint16_t* p = A + t * lda + col;
  if (col + 8 <= d) {
    v = *reinterpret_cast<const u32x4_t*>(p);
  } else if (col < d) {
    uint32_t h[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) h[c] = (col + c < d) ? p[c] : 0u;
    v.x = h[0] | (h[1] << 16);
    v.y = h[2] | (h[3] << 16);
    v.z = h[4] | (h[5] << 16);
    v.w = h[6] | (h[7] << 16);
  }
  return v;
}

// Load the 8 x 8 block (tokens t..t+7, channels col..col+7) into v[8]. Interior blocks take
// eight unconditional 16-byte loads; blocks at the token or channel edge are zero-filled.
__device__ __forceinline__ void load_block(u32x4_t v[8], const uint16_t* __restrict__ A,
                                           int64_t lda, int64_t t, int64_t t_end, int64_t col,
                                           int64_t d) {
  if (t + 8 <= t_end && col + 8 <= d) {
    const uint16_t* p = A + t * lda + col;
#pragma unroll
    for (int r = 0; r < 8; ++r) v[r] = *reinterpret_cast<const u32x4_t*>(p + r * lda);
  } else {
#pragma unroll
    for (int r = 0; r < 8; ++r) v[r] = load_row8(A, lda, t + r, t_end, col, d);
  }
}

// Transpose the block in registers and store channel c's 8 tokens to LDS row (rowbase + c).
__device__ __forceinline__ void store_block_t(uint32_t* __restrict__ lds, const u32x4_t v[8],
                                              int rowbase, int dw_off) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int k = c >> 1;
    const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
    u32x4_t o;
    // dword m packs tokens (2m, 2m+1) of channel c: low half from row 2m, high half from 2m+1
    o.x = __builtin_amdgcn_perm(v[1][k], v[0][k], sel);
    o.y = __builtin_amdgcn_perm(v[3][k], v[2][k], sel);
    o.z = __builtin_amdgcn_perm(v[5][k], v[4][k], sel);
    o.w = __builtin_amdgcn_perm(v[7][k], v[6][k], sel);
    *reinterpret_cast<u32x4_t*>(lds + (rowbase + c) * LROW + dw_off) = o;
  }
}

// Partial tiles are stored in MFMA-fragment order: for wave w (quadrant rows 128 (w % 2), columns
// 128 (w / 2)), accumulator block (bi, bj) and quarter q, lane l's four values (rows
// 8 q + 4 (l / 32) + 0..3 of column l % 32 of the block) are 16 consecutive bytes, and a wave's 64
// lanes one contiguous kilobyte: 64 16-byte stores a lane instead of 256 4-byte ones (the
// stores of a tile measured 5% of the covariance when row-major).
__device__ __forceinline__ void store_partial(float* __restrict__ out, const f32x16_t (&acc)[4][4],
                                              int wave, int lane) {
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int bj = 0; bj < 4; ++bj)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        reinterpret_cast<float4*>(out)[((wave * 4 + bi) * 4 + bj) * 256 + q * 64 + lane] =
            make_float4(acc[bi][bj][4 * q], acc[bi][bj][4 * q + 1], acc[bi][bj][4 * q + 2],
                        acc[bi][bj][4 * q + 3]);
}

template <bool CROSS>
__device__ __forceinline__ void gram_partial(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ B, int64_t tok0,
    int64_t tok_end, int64_t d, int64_t lda, float* __restrict__ part, int n_slices,
    int64_t rows_per_slice, int T, int edge_only, int out_slice0) {
  __shared__ uint32_t lds[2 * 2 * OPER];  // [buffer][operand][256 rows][36 dwords]

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int slice = blockIdx.x % n_slices;
  int I, J;
  if (edge_only) {  // tiles of the last (ragged) block: (I, T-1), I = 0..T-1 (and for cross
                    // also (T-1, J), J = 0..T-2)
    const int e = blockIdx.x / n_slices;
    if (CROSS && e >= T) {
      I = T - 1;
      J = e - T;
    } else {
      I = e;
      J = T - 1;
    }
  } else if (CROSS) {
    const int rem = blockIdx.x / n_slices;
    I = rem / T;
    J = rem % T;
  } else {
    int rem = blockIdx.x / n_slices;
    I = 0;
    while (rem >= T - I) {
      rem -= T - I;
      ++I;
    }
    J = I + rem;
  }
  const int64_t pos =
      CROSS ? int64_t(I) * T + J : int64_t(I) * T - int64_t(I) * (I - 1) / 2 + (J - I);
  const bool diag = !CROSS && (I == J);
  const uint16_t* const Bm = CROSS ? B : A;
  const int64_t i0 = int64_t(I) * TT, j0 = int64_t(J) * TT;
  const int64_t t_begin = tok0 + int64_t(slice) * rows_per_slice;
  const int64_t t_end = min(tok_end, t_begin + rows_per_slice);
  const int64_t n_st = t_end > t_begin ? cdiv(t_end - t_begin, KC) : 0;

  // loader role: token group tg (8 tokens), channel group ig (8 channels)
  const int tg = lane & 7;
  const int ig = wave * 8 + (lane >> 3);
  // compute role
  const int wm = wave & 1, wn = wave >> 1;
  const int l32 = lane & 31, lhi = lane >> 5;

  f32x16_t acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x16_t{};

  u32x4_t va[8], vb[8];
  if (n_st > 0) {
    load_block(va, A, lda, t_begin + tg * 8, t_end, i0 + ig * 8, d);
    if (!diag) load_block(vb, Bm, lda, t_begin + tg * 8, t_end, j0 + ig * 8, d);
    store_block_t(lds, va, ig * 8, tg * 4);
    if (!diag) store_block_t(lds + OPER, vb, ig * 8, tg * 4);
  }
  __syncthreads();

  // MFMA operand fragments, double-buffered across the 16-token steps of a stage so that the
  // LDS reads of step ks+1 are in flight while the 16 MFMAs of step ks run
  bf16x8_t fa[2][4], fb[2][4];
  auto frags = [&](const uint32_t* sa, const uint32_t* sb, int ks, int slot) {
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
      fa[slot][bi] = *reinterpret_cast<const bf16x8_t*>(
          sa + (wm * 128 + bi * 32 + l32) * LROW + ks * 8 + lhi * 4);
#pragma unroll
    for (int bj = 0; bj < 4; ++bj)
      fb[slot][bj] = *reinterpret_cast<const bf16x8_t*>(
          sb + (wn * 128 + bj * 32 + l32) * LROW + ks * 8 + lhi * 4);
  };

  for (int64_t st = 0; st < n_st; ++st) {
    const int buf = int(st & 1);
    const bool more = st + 1 < n_st;
    if (more) {
      const int64_t t = t_begin + (st + 1) * KC + tg * 8;
      load_block(va, A, lda, t, t_end, i0 + ig * 8, d);
      if (!diag) load_block(vb, Bm, lda, t, t_end, j0 + ig * 8, d);
    }
    const uint32_t* sa = lds + buf * 2 * OPER;
    const uint32_t* sb = diag ? sa : sa + OPER;
    frags(sa, sb, 0, 0);
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
      if (ks + 1 < KC / 16) frags(sa, sb, ks + 1, (ks + 1) & 1);
      // keep the next step's LDS reads ahead of this step's MFMAs (the scheduler would
      // otherwise sink each read next to its first use and expose its latency)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int bi = 0; bi < 4; ++bi)
#pragma unroll
        for (int bj = 0; bj < 4; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ks & 1][bi], fb[ks & 1][bj],
                                                                acc[bi][bj], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (more) {
      uint32_t* dst = lds + (buf ^ 1) * 2 * OPER;
      store_block_t(dst, va, ig * 8, tg * 4);
      if (!diag) store_block_t(dst + OPER, vb, ig * 8, tg * 4);
    }
    __syncthreads();
  }

  // the partial tile, in fragment order (store_partial)
  const int64_t npos = CROSS ? int64_t(T) * T : int64_t(T) * (T + 1) / 2;
  store_partial(part + (int64_t(out_slice0 + slice) * npos + pos) * (TT * TT), acc, wave, lane);
}


// ---- interior tiles: direct-to-LDS loads and transposing LDS reads ---------------------------
// Stage = 32 tokens x 256 channels per operand (16 KB), kept in a ring of 4 LDS buffers filled by
// global_load_lds_dwordx4 (64 lanes x 16 bytes straight into LDS, no VGPR staging), so loads run
// three stages ahead. The LDS image is token-major with the 16-byte chunk c8 of token row t
// stored at position c8 ^ (4 (t & 3)); this spreads the rows a transposing read touches over all
// banks. An MFMA operand (32 channels x 8 tokens per lane) is two ds_read_b64_tr_b16: within a
// group of 16 lanes, lane L names token row tb + L/4 at channels cb + 4 (L % 4) .. +3 and gets
// back its own channel cb + L at tokens tb .. tb+3.
// Schedule. A stage is two half-stages of 16 tokens; each half-stage is 16 MFMAs on operands read
// during the previous half-stage, with the next half-stage's 16 reads issued two per MFMA over
// its first eight MFMAs. Between the two halves of stage s, one raw s_barrier (after this wave's
// own loads of stage s + 1 have landed, s_waitcnt vmcnt) both publishes stage s + 1 and frees
// the buffer of stage s - 1. Stage s + 3's loads go out in two parts: its first operand in the
// second half of stage s (into the buffer just freed), its second operand in the first half of
// stage s + 1. The steady state is unrolled
// over the four buffers with every index a constant and no branch, so the compiler places only
// the waits the data needs; the last few stages run a checked copy of the same schedule.
// A diagonal tile loads its block into both operand rings so that no buffer is chosen at run
// time (which would force full waits on every load).
typedef short v4s_t __attribute__((ext_vector_type(4)));
#define KQ_LDS(p) ((__attribute__((address_space(3))) void*)(p))
constexpr int DK = 32;        // tokens per stage
constexpr int RING = 4;       // stage buffers per operand
static_assert(RING == 4, "four stage buffers: the steady state is unrolled over them");
constexpr int PJ = 4;         // tile columns per panel of the tile order
constexpr int SBUF = 4096;    // dwords per operand per stage

template <int N>
__device__ __forceinline__ void wait_vm() {
  // s_waitcnt vmcnt(N) with expcnt / lgkmcnt left unconstrained (gfx9 encoding)
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ bf16x8_t tr_frag(const uint32_t* buf, int tb, int cb, int lane) {
  const int L = lane & 15, g = (lane >> 4) & 1, kh = lane >> 5;
  const int c8 = (cb + g * 16 + 4 * (L & 3)) >> 3;
  v4s_t r[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int t = tb + kh * 8 + h * 4 + (L >> 2);
    const int byte = t * 512 + ((c8 ^ (4 * (t & 3))) << 4) + 8 * (L & 1);
    r[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4s_t*)((const char*)buf + byte));
  }
  bf16x8_t out;
  __builtin_memcpy(&out, r, 16);
  return out;
}

template <bool CROSS>
__device__ __forceinline__ void gram_dma(const uint16_t* __restrict__ A,
                                         const uint16_t* __restrict__ B,
                                         int64_t n_rows, int64_t lda,
                                                        float* __restrict__ part, int n_slices,
                                                        int64_t rows_per_slice, int T, int Tf,
                                                        int n_items) {
  __shared__ __attribute__((aligned(16))) uint32_t a0[SBUF], a1[SBUF], a2[SBUF], a3[SBUF];
  __shared__ __attribute__((aligned(16))) uint32_t b0[SBUF], b1[SBUF], b2[SBUF], b3[SBUF];
  uint32_t* const bufa[RING] = {a0, a1, a2, a3};
  uint32_t* const bufb[RING] = {b0, b1, b2, b3};
  const int tid_launch = threadIdx.x;
  // work items b = blockIdx.x, + gridDim.x, ...: one per workgroup unless the launch caps its
  // workgroups (gridDim.x a multiple of 8 then, so that b % 8 stays the workgroup's XCD)
  for (int item = int(blockIdx.x); item < n_items; item += int(gridDim.x)) {
  // an opaque copy of the thread index per item: the lane-dependent addresses are then formed
  // inside the loop, not hoisted out of it into hundreds of live (spilled) registers
  int tid = tid_launch;
  asm volatile("" : "+v"(tid));
  const int wave = tid >> 6, lane = tid & 63;
  // work item: with S a multiple of 8, XCD x = b % 8 (workgroups are dealt round-robin over the
  // 8 XCDs) runs the tiles of its slices x, x + 8, ... one slice after another, so the
  // workgroups that run together on an XCD read the same tokens through its L2; otherwise
  // slice = b % S
  const int ntile = CROSS ? Tf * Tf : Tf * (Tf + 1) / 2;
  int slice, rem;
  if ((n_slices & 7) == 0) {
    const int kk = item >> 3;
    slice = (kk / ntile) * 8 + (item & 7);
    rem = kk % ntile;
  } else {
    slice = item % n_slices;
    rem = item / n_slices;
  }
  // tile (I <= J; any I, J for cross) of sequence number rem: panels of PJ tile columns, within
  // a panel by rows, so that the 32 workgroups running together on an XCD form an 8 x 4 block of
  // tiles that reads 12 channel blocks rather than up to 64 (at d = 28672 this cut the time by
  // 9-11%)
  int I, J;
  if (CROSS) {
    const int pp = rem / (Tf * PJ), r = rem % (Tf * PJ);
    const int j0 = pp * PJ, w = min(Tf, j0 + PJ) - j0;
    I = r / w;
    J = j0 + r % w;
  } else {
    int pp = 0, r = rem;
    while (true) {
      const int j0 = pp * PJ, w = min(Tf, j0 + PJ) - j0;
      const int cnt = j0 * w + w * (w + 1) / 2;
      if (r < cnt) break;
      r -= cnt;
      ++pp;
    }
    const int j0 = pp * PJ, w = min(Tf, j0 + PJ) - j0;
    if (r < j0 * w) {
      I = r / w;
      J = j0 + r % w;
    } else {
      r -= j0 * w;
      int i = 0;
      while (r >= w - i) {
        r -= w - i;
        ++i;
      }
      I = j0 + i;
      J = I + r;
    }
  }
  const int64_t pos =
      CROSS ? int64_t(I) * T + J : int64_t(I) * T - int64_t(I) * (I - 1) / 2 + (J - I);
  const int64_t t_begin = int64_t(slice) * rows_per_slice;
  const int64_t t_end = min(n_rows, t_begin + rows_per_slice);
  const int n_st = t_end > t_begin ? int((t_end - t_begin) / DK) : 0;  // full stages
  int64_t off[4];  // this lane's source offsets (elements) for its 4 chunks per operand
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int q = (wave * 4 + k) * 64 + lane;
    const int t = q >> 5, c8 = (q & 31) ^ (4 * (t & 3));
    off[k] = int64_t(t) * lda + 8 * c8;
  }
  const uint16_t* Ai = A + t_begin * lda + int64_t(I) * TT;
  const uint16_t* Aj = (CROSS ? B : A) + t_begin * lda + int64_t(J) * TT;
  // this wave's 4 loads of one operand (part 0: rows I, part 1: rows J) of stage st
  auto issue_part = [&](int st, int b, int part) {
    const int64_t so = int64_t(st) * DK * lda;
    const uint16_t* src = part ? Aj : Ai;
    uint32_t* dst = part ? bufb[b] : bufa[b];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      __builtin_amdgcn_global_load_lds(src + so + off[k], KQ_LDS(dst + (wave * 4 + k) * 256), 16,
                                       0, 0);
  };
  auto issue = [&](int st, int b) {
    issue_part(st, b, 0);
    issue_part(st, b, 1);
  };
  const int wm = wave & 1, wn = wave >> 1;
  f32x16_t acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = f32x16_t{};
  bf16x8_t fa[2][4], fb[2][4];
  auto frags = [&](int b, int ks, int slot) {
#pragma unroll
    for (int bi = 0; bi < 4; ++bi) fa[slot][bi] = tr_frag(bufa[b], ks * 16, wm * 128 + bi * 32, lane);
#pragma unroll
    for (int bj = 0; bj < 4; ++bj) fb[slot][bj] = tr_frag(bufb[b], ks * 16, wn * 128 + bj * 32, lane);
  };
  auto mfmas = [&](int slot) {
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int bj = 0; bj < 4; ++bj)
        acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][bi], fb[slot][bj],
                                                              acc[bi][bj], 0, 0, 0);
  };
  // this wave's loads of stage s + 1 are done when at most `newer` later stages are pending
  auto wait_newer = [&](int newer) {
    if (newer >= 3) wait_vm<24>();
    else if (newer == 2) wait_vm<16>();
    else if (newer == 1) wait_vm<8>();
    else wait_vm<0>();
  };
  // steady state: stage s issues the rest of stage s + RING - 2 and the first half of stage
  // s + RING - 1 unconditionally, no branches inside
  const int s_main = n_st >= 2 * RING - 1 ? ((n_st - RING + 1) / RING) * RING : 0;
  if (n_st > 0) {
    if (s_main > 0) {  // stages 0 .. RING - 3, and the first operand of stage RING - 2
#pragma unroll
      for (int p = 0; p < RING - 2; ++p) issue(p, p);
      issue_part(RING - 2, RING - 2, 0);
      wait_vm<(RING - 3) * 8 + 4>();
    } else {
#pragma unroll
      for (int p = 0; p < RING - 1; ++p)
        if (p < n_st) issue(p, p);
      wait_newer(min(RING - 2, n_st - 1));
    }
    __builtin_amdgcn_s_barrier();
    frags(0, 0, 0);
  }
  // Each half-stage: 16 MFMAs; the next half-stage's 16 operand reads two per MFMA over the
  // first 8 (a use of a transposing read's result waits for every outstanding LDS read, so all
  // must have landed by the next half-stage); 4 global-to-LDS loads over the last 8, one per two
  // MFMAs. A stage's 8 loads are
  // split over two half-stages (all 8 in one burst of 8 MFMAs queued behind each other in the
  // address unit and held up the MFMAs behind them).
  auto pattern = [&]() {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // two LDS reads
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one global-to-LDS load
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    }
  };
  auto body = [&](auto ucst, int s) {
    constexpr int u = decltype(ucst)::value;
    __builtin_amdgcn_sched_barrier(0);
    // first half-stage: the second operand of stage s + 2 (its buffer, that of stage s - 2, has
    // been free since the barrier of stage s - 1)
    issue_part(s + RING - 2, (u + RING - 2) % RING, 1);
    frags(u, 1, 1);
    mfmas(0);
    pattern();
    __builtin_amdgcn_sched_barrier(0);
    // this wave's loads of stage s + 1 have landed when only those of stages s + 2 ..
    // s + RING - 2 are newer
    wait_vm<(RING - 3) * 8>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // second half-stage: the first operand of stage s + 3 into the buffer of stage s - 1, whose
    // last reads every wave finished before this barrier
    issue_part(s + RING - 1, (u + RING - 1) % RING, 0);
    frags((u + 1) % RING, 0, 0);
    mfmas(1);
    pattern();
    __builtin_amdgcn_sched_barrier(0);
  };
  for (int s0 = 0; s0 < s_main; s0 += RING) {
    body(std::integral_constant<int, 0>{}, s0);
    body(std::integral_constant<int, 1>{}, s0 + 1);
    body(std::integral_constant<int, 2>{}, s0 + 2);
    body(std::integral_constant<int, 3>{}, s0 + 3);
  }
  // the second operand of stage s_main + RING - 2 (< n_st), so that the tail finds whole stages
  // issued
  if (s_main > 0) issue_part(s_main + RING - 2, (s_main + RING - 2) % RING, 1);
  // tail (the last few stages), with the bounds checks
  for (int s0 = s_main; s0 < n_st; s0 += RING) {
#pragma unroll
    for (int u = 0; u < RING; ++u) {
      const int s = s0 + u;  // stage s lives in buffer u
      if (s < n_st) {
        frags(u, 1, 1);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(0);
        __builtin_amdgcn_sched_barrier(0);
        if (s + 1 < n_st) {
          const int last = min(n_st - 1, s + RING - 2);  // newest stage already issued
          wait_newer(last - (s + 1));
          __builtin_amdgcn_s_barrier();
          if (s + RING - 1 < n_st) issue(s + RING - 1, (u + RING - 1) % RING);
          frags((u + 1) % RING, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        mfmas(1);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  const int64_t npos = CROSS ? int64_t(T) * T : int64_t(T) * (T + 1) / 2;
  store_partial(part + (int64_t(slice) * npos + pos) * (TT * TT), acc, wave, lane);
  __syncthreads();  // the ring's last reads are done before the next item's loads overwrite it
  }
}

// Sum the S partial tiles of one 64 x 64 sub-block and write H (and its mirror; cross: the
// sub-block as it is). The sub-block is 2 x 2 accumulator blocks of one wave's quadrant: thread
// (block b, lane) reads that lane's four 16-byte quarters of each partial tile (a wave's loads of
// one quarter are one contiguous kilobyte), adds the slices in order, and the sums pass through
// LDS so that both H and its mirror are written in whole rows.
template <bool CROSS>
__device__ __forceinline__ void gram_reduce(const float* __restrict__ part, int n_slices, int T,
                                            int64_t d, float* __restrict__ H, int64_t ldh,
                                            float alpha, float beta) {
  __shared__ float tr[64][65];
  const int pos = blockIdx.x >> 4;
  const int sub = blockIdx.x & 15;
  int I = 0, J = 0;
  if (CROSS) {
    I = pos / T;
    J = pos % T;
  } else {
    int rem = pos;
    while (rem >= T - I) {
      rem -= T - I;
      ++I;
    }
    J = I + rem;
  }
  const int sr = (sub >> 2) * 64, sc = (sub & 3) * 64;  // sub-block origin inside the tile
  // below the diagonal of a diagonal tile nothing is written here (the mirror comes from the
  // sub-block across the diagonal)
  if (!CROSS && I == J && sr > sc) return;
  const int64_t gi0 = int64_t(I) * TT + sr, gj0 = int64_t(J) * TT + sc;
  const int64_t npos = CROSS ? int64_t(T) * T : int64_t(T) * (T + 1) / 2;
  const int tid = threadIdx.x, lane = tid & 63, b = tid >> 6;
  const int w = (sr >> 7) + 2 * (sc >> 7);  // the wave whose quadrant holds the sub-block
  const int bi = ((sr & 127) >> 5) + (b >> 1), bj = ((sc & 127) >> 5) + (b & 1);
  const float4* base = reinterpret_cast<const float4*>(part + int64_t(pos) * (TT * TT)) +
                       ((w * 4 + bi) * 4 + bj) * 256 + lane;
  const int64_t slice4 = npos * (TT * TT / 4);
  // slices added in order; four slices of the four quarters (16 loads) in flight at a time
  float4 v[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] = make_float4(0.f, 0.f, 0.f, 0.f);
  int s = 0;
  for (; s + 4 <= n_slices; s += 4) {
    float4 x[4][4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int u = 0; u < 4; ++u) x[q][u] = base[(s + u) * slice4 + q * 64];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v[q].x += x[q][u].x;
        v[q].y += x[q][u].y;
        v[q].z += x[q][u].z;
        v[q].w += x[q][u].w;
      }
  }
  for (; s < n_slices; ++s) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 x = base[s * slice4 + q * 64];
      v[q].x += x.x;
      v[q].y += x.y;
      v[q].z += x.z;
      v[q].w += x.w;
    }
  }
  // quarter q, element e of this lane: row 8 q + 4 (lane / 32) + e, column lane % 32 of its block
  {
    const int rl = (b >> 1) * 32 + 4 * (lane >> 5), cl = (b & 1) * 32 + (lane & 31);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      tr[rl + 8 * q][cl] = v[q].x;
      tr[rl + 8 * q + 1][cl] = v[q].y;
      tr[rl + 8 * q + 2][cl] = v[q].z;
      tr[rl + 8 * q + 3][cl] = v[q].w;
    }
  }
  __syncthreads();
  // the sub-block in rows (cross: all of it; syrk: the upper triangle, i <= j)
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int idx = tid + 256 * k;
    const int ii = idx >> 6, jj = idx & 63;
    const int64_t gi = gi0 + ii, gj = gj0 + jj;
    if (gi < d && gj < d && (CROSS || gi <= gj)) {
      float* h = H + gi * ldh + gj;
      const float x = tr[ii][jj];
      *h = beta == 0.f ? alpha * x : alpha * x + beta * *h;
    }
  }
  if (CROSS) return;
  // mirror: H[j][i] = value of (i, j) for i < j, coalesced along i; the strict lower triangle
  // is the upper one's mirror, so H is exactly symmetric (diagonal tiles included)
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int idx = tid + 256 * k;
    const int jj = idx >> 6, ii = idx & 63;
    const int64_t gj = gj0 + jj, gi = gi0 + ii;
    if (gi < d && gj < d && gi < gj) {
      float* h = H + gj * ldh + gi;
      const float x = tr[ii][jj];
      *h = beta == 0.f ? alpha * x : alpha * x + beta * *h;
    }
  }
}

// One kernel name per product, so that traces and profiles tell the two apart.
#define KQ_GRAM_PARTIAL_ARGS                                                                    \
  const uint16_t *__restrict__ A, const uint16_t *__restrict__ B, int64_t tok0, int64_t tok_end, \
      int64_t d, int64_t lda, float *__restrict__ part, int n_slices, int64_t rows_per_slice,    \
      int T, int edge_only, int out_slice0
__global__ __launch_bounds__(256, 1) void syrk_bf16_partial(KQ_GRAM_PARTIAL_ARGS) {
  gram_partial<false>(A, B, tok0, tok_end, d, lda, part, n_slices, rows_per_slice, T, edge_only,
                      out_slice0);
}
__global__ __launch_bounds__(256, 1) void cross_bf16_partial(KQ_GRAM_PARTIAL_ARGS) {
  gram_partial<true>(A, B, tok0, tok_end, d, lda, part, n_slices, rows_per_slice, T, edge_only,
                     out_slice0);
}
#define KQ_GRAM_DMA_ARGS                                                                  \
  const uint16_t *__restrict__ A, const uint16_t *__restrict__ B, int64_t n_rows, int64_t lda, \
      float *__restrict__ part, int n_slices, int64_t rows_per_slice, int T, int Tf, int n_items
__global__ __launch_bounds__(256, 1) void syrk_bf16_dma(KQ_GRAM_DMA_ARGS) {
  gram_dma<false>(A, B, n_rows, lda, part, n_slices, rows_per_slice, T, Tf, n_items);
}
// the same kernel for a launch that holds part of the chip (its own name in profiles)
__global__ __launch_bounds__(256, 1) void syrk_bf16_dma_shared(KQ_GRAM_DMA_ARGS) {
  gram_dma<false>(A, B, n_rows, lda, part, n_slices, rows_per_slice, T, Tf, n_items);
}
__global__ __launch_bounds__(256, 1) void cross_bf16_dma(KQ_GRAM_DMA_ARGS) {
  gram_dma<true>(A, B, n_rows, lda, part, n_slices, rows_per_slice, T, Tf, n_items);
}
#define KQ_GRAM_REDUCE_ARGS                                                                \
  const float *__restrict__ part, int n_slices, int T, int64_t d, float *__restrict__ H,   \
      int64_t ldh, float alpha, float beta
__global__ __launch_bounds__(256) void syrk_reduce(KQ_GRAM_REDUCE_ARGS) {
  gram_reduce<false>(part, n_slices, T, d, H, ldh, alpha, beta);
}
__global__ __launch_bounds__(256) void cross_reduce(KQ_GRAM_REDUCE_ARGS) {
  gram_reduce<true>(part, n_slices, T, d, H, ldh, alpha, beta);
}
#undef KQ_GRAM_PARTIAL_ARGS
#undef KQ_GRAM_DMA_ARGS
#undef KQ_GRAM_REDUCE_ARGS

// Plain fp32 A^T B for fp32 inputs (B = A for the covariance): 64 x 64 tiles, 4 x 4 outputs per
// thread.
__global__ __launch_bounds__(256) void syrk_f32(const float* __restrict__ A,
                                                const float* __restrict__ B, int64_t n_rows,
                                                int64_t d, int64_t lda, float* __restrict__ H,
                                                int64_t ldh, float alpha, float beta) {
  __shared__ float sa[16][64];
  __shared__ float sb[16][64];
  const int tid = threadIdx.x;
  const int64_t i0 = int64_t(blockIdx.y) * 64, j0 = int64_t(blockIdx.x) * 64;
  const int ti = (tid >> 4) * 4, tj = (tid & 15) * 4;
  float acc[4][4] = {};
  for (int64_t t0 = 0; t0 < n_rows; t0 += 16) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int idx = tid + 256 * k;
      const int r = idx >> 6, c = idx & 63;
      const int64_t t = t0 + r;
      sa[r][c] = (t < n_rows && i0 + c < d) ? A[t * lda + i0 + c] : 0.f;
      sb[r][c] = (t < n_rows && j0 + c < d) ? B[t * lda + j0 + c] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float a[4], b[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = sa[r][ti + e];
        b[e] = sb[r][tj + e];
      }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = fmaf(a[x], b[y], acc[x][y]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const int64_t i = i0 + ti + x, j = j0 + tj + y;
      if (i < d && j < d) {
        float* h = H + i * ldh + j;
        *h = beta == 0.f ? alpha * acc[x][y] : alpha * acc[x][y] + beta * *h;
      }
    }
}

// H <- beta H (no tokens)
__global__ void scale_matrix(float* __restrict__ H, int64_t d, int64_t ldh, float beta) {
  const int64_t i = blockIdx.y;
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < d;
       j += int64_t(gridDim.x) * blockDim.x) {
    float* h = H + i * ldh + j;
    *h = beta == 0.f ? 0.f : beta * *h;
  }
}

struct CovPlan {
  int T = 0;    // 256-channel blocks (the last may be ragged)
  int Tf = 0;   // full 256-channel blocks
  int S = 0;    // token slices (one per XCD when there are enough tokens)
  int64_t rows_per_slice = 0;
  int64_t npos = 0;
  int64_t tail_begin = 0;  // tokens [tail_begin, n_rows) do not fill a 32-token stage
  bool tail = false;
};


// Token slices S (split-K). Each interior tile x slice is one workgroup holding a whole CU, so
// the launch runs in ceil(W / CUs) rounds of equal length for W = tiles * S workgroups; the
// last round is partly idle unless W fills it. Each slice also costs one partial tile per tile
// to write and to reduce, worth about 500 tokens of that tile's MFMA time (256 KB at HBM speed
// against 256 x 256 x 2 flops per token at MFMA speed). S minimises
//   ceil(W / CUs) * CUs / W + 500 S / N
// over the multiples of 8 up to 32 (which keep each XCD on its own slices; other counts mix
// token ranges on an XCD and measured slower), or 1..7 when there are too few tokens for 8
// slices of 4 * KC. At d = 4096, N = 262144 this gives S = 32: 4352 workgroups in exactly 17
// rounds, instead of S = 8 in 4.25 rounds. A launch capped to part of the chip counts rounds of
// its own persistent workgroups (cus_avail): on 128 CUs the same covariance takes S = 16,
// 2176 items in 17 rounds, with half the partial tiles to write and to reduce.
CovPlan cov_plan(int64_t n_rows, int64_t d, bool cross, int64_t cus_avail = 0) {
  CovPlan p;
  p.T = int(cdiv(d, TT));
  p.Tf = int(d / TT);
  p.npos = cross ? int64_t(p.T) * p.T : int64_t(p.T) * (p.T + 1) / 2;
  const int64_t full = cross ? int64_t(p.Tf) * p.Tf : int64_t(p.Tf) * (p.Tf + 1) / 2;
  const int64_t tiles = full > 0 ? full : p.npos;
  const int64_t smax = std::max<int64_t>(1, std::min<int64_t>(32, n_rows / (4 * KC)));
  const double cus = double(cus_avail > 0 ? cus_avail : device_cus());
  double best = 1e300;
  // multiples of 8 whenever the tokens allow it (they keep each XCD on its own slices, which
  // the cost model does not price); 1..7 only for short inputs
  for (int64_t S = smax >= 8 ? 8 : 1; S <= smax; S += (S < 8 ? 1 : 8)) {
    const double W = double(tiles * S);
    const double cost = std::ceil(W / cus) * cus / W + 500.0 * double(S) / double(n_rows);
    if (cost < best - 1e-12) {
      best = cost;
      p.S = int(S);
    }
  }
  p.rows_per_slice = cdiv(cdiv(n_rows, p.S), KC) * KC;
  // rounding the slice up to whole stages can leave trailing slices empty: keep only the
  // non-empty ones, so that every slice but the last is full and the last starts before n_rows
  p.S = int(cdiv(n_rows, p.rows_per_slice));
  const int64_t last = int64_t(p.S - 1) * p.rows_per_slice;
  const int64_t in_last = n_rows > last ? n_rows - last : 0;
  p.tail_begin = last + (in_last / DK) * DK;
  p.tail = p.tail_begin < n_rows;
  return p;
}

// the bf16 pipeline shared by the covariance (B == nullptr) and the cross product
// max_cus > 0: the interior-tile launch holds at most that many CUs at once (persistent
// workgroups, one per CU, a multiple of 8), leaving the rest of the chip to other streams
int gram_bf16(const uint16_t* A, const uint16_t* B, int64_t n_rows, int64_t d, int64_t lda,
              float* H, int64_t ldh, float alpha, float beta, void* ws, int max_cus,
              hipStream_t s) {
  const bool cross = B != nullptr;
  CovPlan p = cov_plan(n_rows, d, cross);
  if (max_cus > 0 && max_cus < device_cus()) {
    // persistent workgroups on part of the chip: the slices that fill whole rounds of them (the
    // workspace holds the whole-chip plan's slices, so only a plan with no more is taken)
    const CovPlan q = cov_plan(n_rows, d, cross, max_cus >= 8 ? (max_cus / 8) * 8 : max_cus);
    if (q.S <= p.S) p = q;
  }
  float* part = static_cast<float*>(ws);
  const int64_t full = cross ? int64_t(p.Tf) * p.Tf : int64_t(p.Tf) * (p.Tf + 1) / 2;
  // interior tiles, whole 32-token stages of every slice
  if (p.Tf > 0) {
    const int64_t items = int64_t(p.S) * full;
    int64_t wgs = items;
    if (max_cus > 0 && items > max_cus) wgs = max_cus >= 8 ? (max_cus / 8) * 8 : max_cus;
    const dim3 grid(static_cast<unsigned>(wgs));
    if (cross)
      KQ_TRY(launch("cross_bf16_mfma", cross_bf16_dma, grid, dim3(256), 0, s, A, B, n_rows,
                    lda, part, p.S, p.rows_per_slice, p.T, p.Tf, int(items)));
    else if (wgs < items)
      KQ_TRY(launch("syrk_bf16_mfma_shared", syrk_bf16_dma_shared, grid, dim3(256), 0, s, A, A,
                    n_rows, lda, part, p.S, p.rows_per_slice, p.T, p.Tf, int(items)));
    else
      KQ_TRY(launch("syrk_bf16_mfma", syrk_bf16_dma, grid, dim3(256), 0, s, A, A, n_rows,
                    lda, part, p.S, p.rows_per_slice, p.T, p.Tf, int(items)));
  }
  // tiles of a ragged last channel block, same tokens
  const int64_t body_end = p.tail ? p.tail_begin : n_rows;
  if (p.T > p.Tf) {
    const dim3 grid(unsigned(p.S * (cross ? 2 * p.T - 1 : p.T)));
    if (cross)
      KQ_TRY(launch("cross_bf16_edge", cross_bf16_partial, grid, dim3(256), 0, s, A, B,
                    int64_t(0), body_end, d, lda, part, p.S, p.rows_per_slice, p.T, 1, 0));
    else
      KQ_TRY(launch("syrk_bf16_edge", syrk_bf16_partial, grid, dim3(256), 0, s, A, A,
                    int64_t(0), body_end, d, lda, part, p.S, p.rows_per_slice, p.T, 1, 0));
  }
  // the last < 32 tokens, every tile, as one extra slice
  if (p.tail) {
    const dim3 grid(unsigned(p.npos));
    if (cross)
      KQ_TRY(launch("cross_bf16_tail", cross_bf16_partial, grid, dim3(256), 0, s, A, B,
                    p.tail_begin, n_rows, d, lda, part, 1, n_rows - p.tail_begin, p.T, 0, p.S));
    else
      KQ_TRY(launch("syrk_bf16_tail", syrk_bf16_partial, grid, dim3(256), 0, s, A, A,
                    p.tail_begin, n_rows, d, lda, part, 1, n_rows - p.tail_begin, p.T, 0, p.S));
  }
  const int ns = p.S + (p.tail ? 1 : 0);
  if (cross)
    return launch("cross_reduce", cross_reduce, dim3(unsigned(p.npos * 16)), dim3(256), 0, s,
                  static_cast<const float*>(part), ns, p.T, d, H, ldh, alpha, beta);
  return launch("syrk_reduce", syrk_reduce, dim3(unsigned(p.npos * 16)), dim3(256), 0, s,
                static_cast<const float*>(part), ns, p.T, d, H, ldh, alpha, beta);
}

}  // namespace

size_t cov_ws_bytes(int dtype, int64_t n_rows, int64_t d, bool cross) {
  if (dtype != KRONQ_BF16 || n_rows <= 0 || d <= 0) return 0;
  const CovPlan p = cov_plan(n_rows, d, cross);
  return align256(size_t(p.S + 1) * size_t(p.npos) * TT * TT * sizeof(float));
}

int cov_launch(const void* A, const void* B, int dtype, int64_t n_rows, int64_t d, int64_t lda,
               float* H, int64_t ldh, float alpha, float beta, void* ws, hipStream_t s,
               int max_cus) {
  if (n_rows == 0) {
    return launch("cov_scale", scale_matrix, dim3(unsigned(cdiv(d, 256)), unsigned(d)), dim3(256),
                  0, s, H, d, ldh, beta);
  }
  if (dtype == KRONQ_FP32) {
    const unsigned g = unsigned(cdiv(d, 64));
    const float* a = static_cast<const float*>(A);
    return launch(B ? "cross_f32" : "syrk_f32", syrk_f32, dim3(g, g), dim3(256), 0, s, a,
                  B ? static_cast<const float*>(B) : a, n_rows, d, lda, H, ldh, alpha, beta);
  }
  return gram_bf16(static_cast<const uint16_t*>(A), static_cast<const uint16_t*>(B), n_rows, d,
                   lda, H, ldh, alpha, beta, ws, max_cus, s);
}

}  // namespace kq
