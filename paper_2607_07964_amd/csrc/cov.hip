// Covariance accumulation H <- beta H + alpha A^T A (Sec. 4.1 eq. kfac; Alg. 1 first line).
//
// bf16 path: a syrk on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16). bf16 x bf16 products
// are exact in fp32 and accumulate in fp32.
//   * Work split: the token dimension is cut into S slices (split-K). Workgroup b takes slice
//     b % S, so with S = 8 each XCD (workgroups are dealt round-robin over the 8 XCDs) streams
//     its own eighth of the tokens and every tile on that XCD reuses it through the XCD's L2.
//   * Each workgroup owns one 256 x 256 tile (I <= J) of the upper triangle of H for its slice:
//     4 waves, each a 128 x 128 sub-tile = 4 x 4 MFMA blocks of 32 x 32, 256 fp32
//     accumulators per lane.
//   * Per stage, 64 tokens x 256 columns of each operand are loaded as 8 x 8 bf16 blocks
//     (eight 16-byte loads along the channel axis), transposed in registers with v_perm, and
//     written token-contiguous to LDS with 16-byte stores. An MFMA operand is then a single
//     16-byte LDS read. The LDS row stride of 72 bf16 (36 dwords) makes both the stores and
//     the operand reads conflict-free. LDS is double-buffered: the loads for stage s+1 are in
//     flight while stage s runs, one barrier per stage. A diagonal tile loads one operand.
//   * Partial tiles go to the workspace; a reduction kernel sums the S slices, applies
//     alpha/beta and writes both triangles (the mirror through an LDS transpose).
// fp32 path (small fp32 inputs): a plain LDS-tiled fp32 FMA kernel over the full matrix.
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

// Load the 8 x 8 block (tokens t..t+7, channels col..col+7) into v[8].
__device__ __forceinline__ void load_block(u32x4_t v[8], const uint16_t* __restrict__ A,
                                           int64_t lda, int64_t t, int64_t t_end, int64_t col,
                                           int64_t d) {
#pragma unroll
  for (int r = 0; r < 8; ++r) v[r] = load_row8(A, lda, t + r, t_end, col, d);
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

__global__ __launch_bounds__(256, 1) void syrk_bf16_partial(
    const uint16_t* __restrict__ A, int64_t n_rows, int64_t d, int64_t lda,
    float* __restrict__ part, int n_slices, int64_t rows_per_slice, int T) {
  __shared__ uint32_t lds[2 * 2 * OPER];  // [buffer][operand][256 rows][36 dwords]

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int slice = blockIdx.x % n_slices;
  const int pos = blockIdx.x / n_slices;
  int I = 0, rem = pos;
  while (rem >= T - I) {
    rem -= T - I;
    ++I;
  }
  const int J = I + rem;
  const bool diag = (I == J);
  const int64_t i0 = int64_t(I) * TT, j0 = int64_t(J) * TT;
  const int64_t t_begin = int64_t(slice) * rows_per_slice;
  const int64_t t_end = min(n_rows, t_begin + rows_per_slice);
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
    if (!diag) load_block(vb, A, lda, t_begin + tg * 8, t_end, j0 + ig * 8, d);
    store_block_t(lds, va, ig * 8, tg * 4);
    if (!diag) store_block_t(lds + OPER, vb, ig * 8, tg * 4);
  }
  __syncthreads();

  for (int64_t st = 0; st < n_st; ++st) {
    const int buf = int(st & 1);
    const bool more = st + 1 < n_st;
    if (more) {
      const int64_t t = t_begin + (st + 1) * KC + tg * 8;
      load_block(va, A, lda, t, t_end, i0 + ig * 8, d);
      if (!diag) load_block(vb, A, lda, t, t_end, j0 + ig * 8, d);
    }
    const uint32_t* sa = lds + buf * 2 * OPER;
    const uint32_t* sb = diag ? sa : sa + OPER;
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
      bf16x8_t fa[4], fb[4];
#pragma unroll
      for (int bi = 0; bi < 4; ++bi) {
        const int row = wm * 128 + bi * 32 + l32;
        fa[bi] = *reinterpret_cast<const bf16x8_t*>(sa + row * LROW + ks * 8 + lhi * 4);
      }
#pragma unroll
      for (int bj = 0; bj < 4; ++bj) {
        const int row = wn * 128 + bj * 32 + l32;
        fb[bj] = *reinterpret_cast<const bf16x8_t*>(sb + row * LROW + ks * 8 + lhi * 4);
      }
#pragma unroll
      for (int bi = 0; bi < 4; ++bi)
#pragma unroll
        for (int bj = 0; bj < 4; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[bi], fb[bj], acc[bi][bj], 0, 0, 0);
    }
    if (more) {
      uint32_t* dst = lds + (buf ^ 1) * 2 * OPER;
      store_block_t(dst, va, ig * 8, tg * 4);
      if (!diag) store_block_t(dst + OPER, vb, ig * 8, tg * 4);
    }
    __syncthreads();
  }

  // partial tile, row-major 256 x 256 (rows: channels i of the tile, cols: channels j)
  const int64_t npos = int64_t(T) * (T + 1) / 2;
  float* out = part + (int64_t(slice) * npos + pos) * (TT * TT);
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int bj = 0; bj < 4; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * 128 + bi * 32 + (r >> 2) * 8 + lhi * 4 + (r & 3);
        const int col = wn * 128 + bj * 32 + l32;
        out[row * TT + col] = acc[bi][bj][r];
      }
}

// Sum the S partial tiles of one 64 x 64 sub-block and write H (and its mirror).
__global__ __launch_bounds__(256) void syrk_reduce(const float* __restrict__ part, int n_slices,
                                                   int T, int64_t d, float* __restrict__ H,
                                                   int64_t ldh, float alpha, float beta) {
  __shared__ float tr[64][65];
  const int pos = blockIdx.x >> 4;
  const int sub = blockIdx.x & 15;
  int I = 0, rem = pos;
  while (rem >= T - I) {
    rem -= T - I;
    ++I;
  }
  const int J = I + rem;
  const int sr = (sub >> 2) * 64, sc = (sub & 3) * 64;  // sub-block origin inside the tile
  const int64_t gi0 = int64_t(I) * TT + sr, gj0 = int64_t(J) * TT + sc;
  const int64_t npos = int64_t(T) * (T + 1) / 2;
  const int tid = threadIdx.x;
  const int c4 = (tid & 15) * 4;
  const int rb = tid >> 4;
  float v[4][4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = rb + 16 * k;
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    for (int s = 0; s < n_slices; ++s) {
      const float4 x = *reinterpret_cast<const float4*>(
          part + (int64_t(s) * npos + pos) * (TT * TT) + (sr + r) * TT + sc + c4);
      s0 += x.x;
      s1 += x.y;
      s2 += x.z;
      s3 += x.w;
    }
    v[k][0] = s0;
    v[k][1] = s1;
    v[k][2] = s2;
    v[k][3] = s3;
  }
  // upper triangle (i <= j) from the sums; the strict lower triangle is its mirror, so H is
  // exactly symmetric (diagonal tiles included)
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t gi = gi0 + rb + 16 * k;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t gj = gj0 + c4 + e;
      if (gi < d && gj < d && gi <= gj) {
        float* h = H + gi * ldh + gj;
        *h = beta == 0.f ? alpha * v[k][e] : alpha * v[k][e] + beta * *h;
      }
      tr[c4 + e][rb + 16 * k] = v[k][e];
    }
  }
  __syncthreads();
  // mirror: H[j][i] = value of (i, j) for i < j, coalesced along i
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int idx = tid + 256 * k;
    const int jj = idx >> 6, ii = idx & 63;
    const int64_t gj = gj0 + jj, gi = gi0 + ii;
    if (gi < d && gj < d && gi < gj) {
      float* h = H + gj * ldh + gi;
      const float x = tr[jj][ii];
      *h = beta == 0.f ? alpha * x : alpha * x + beta * *h;
    }
  }
}

// Plain fp32 syrk for fp32 inputs: 64 x 64 tiles, 4 x 4 outputs per thread.
__global__ __launch_bounds__(256) void syrk_f32(const float* __restrict__ A, int64_t n_rows,
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
      sb[r][c] = (t < n_rows && j0 + c < d) ? A[t * lda + j0 + c] : 0.f;
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
  int T = 0;
  int S = 0;
  int64_t rows_per_slice = 0;
  int64_t npos = 0;
};

CovPlan cov_plan(int64_t n_rows, int64_t d) {
  CovPlan p;
  p.T = int(cdiv(d, TT));
  p.npos = int64_t(p.T) * (p.T + 1) / 2;
  // one token slice per XCD when there are enough tokens; fewer slices for short inputs
  int64_t s = n_rows / (4 * KC);
  p.S = int(s < 1 ? 1 : (s > 8 ? 8 : s));
  p.rows_per_slice = cdiv(cdiv(n_rows, p.S), KC) * KC;
  return p;
}

}  // namespace

size_t cov_ws_bytes(int dtype, int64_t n_rows, int64_t d) {
  if (dtype != KRONQ_BF16 || n_rows <= 0 || d <= 0) return 0;
  const CovPlan p = cov_plan(n_rows, d);
  return align256(size_t(p.S) * size_t(p.npos) * TT * TT * sizeof(float));
}

int cov_launch(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda, float* H,
               int64_t ldh, float alpha, float beta, void* ws, hipStream_t s) {
  if (n_rows == 0) {
    return launch("cov_scale", scale_matrix, dim3(unsigned(cdiv(d, 256)), unsigned(d)), dim3(256),
                  0, s, H, d, ldh, beta);
  }
  if (dtype == KRONQ_FP32) {
    const unsigned g = unsigned(cdiv(d, 64));
    return launch("syrk_f32", syrk_f32, dim3(g, g), dim3(256), 0, s,
                  static_cast<const float*>(A), n_rows, d, lda, H, ldh, alpha, beta);
  }
  const CovPlan p = cov_plan(n_rows, d);
  float* part = static_cast<float*>(ws);
  KQ_TRY(launch("syrk_bf16_mfma", syrk_bf16_partial, dim3(unsigned(p.S * p.npos)), dim3(256), 0, s,
                static_cast<const uint16_t*>(A), n_rows, d, lda, part, p.S, p.rows_per_slice,
                p.T));
  return launch("syrk_reduce", syrk_reduce, dim3(unsigned(p.npos * 16)), dim3(256), 0, s,
                static_cast<const float*>(part), p.S, p.T, d, H, ldh, alpha, beta);
}

}  // namespace kq
