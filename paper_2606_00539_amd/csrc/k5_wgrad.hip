// K5, the gradient pass fused into its producer for CDNA4 (gfx950): the
// weight-gradient GEMM of a linear layer with the sum of squares that the
// controller needs computed in its epilogue, so that the gradient is never
// read back from HBM for its norm (the norm is the only per-unit quantity
// the controller takes from the gradient, Sec. 3.3 and Alg. 1; it is cheap
// to compute from what the producer already holds, Sec. 3.1).
//
//   dw[o][i] = bf16_rne( sum_t dy[t][o] * x[t][i] )   fp32 accumulation
//   tile_ss[tile] = sum over the tile of float(dw)^2  fp32, fixed order
//
// dy: [tokens][out] bf16, x: [tokens][in] bf16, dw: [out][in] bf16, all
// row-major.  The contraction runs over the slow (token) index of both
// operands, so both tiles sit in LDS exactly as they arrive ([k][feature],
// features contiguous) and reach the matrix cores through the transposing
// LDS read ds_read_b64_tr_b16, which hands each lane four consecutive k of
// one feature.
//
// Tiling: one 256-lane workgroup per 256x256 output tile, four waves of
// 128x128 (4x4 v_mfma_f32_32x32x16_bf16 blocks each), K steps of 64 with two
// LDS stages: the global loads of step s+1 are in flight while the matrix
// cores work on step s.  x is the matrix cores' A operand, so the four
// accumulator rows a lane holds per group are four consecutive output
// columns: each lane stores 8 contiguous bytes.
#include "gnmr_internal.h"

namespace gnmr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) u32x2 g_vec2;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Buffer resource word 3 for gfx9-family raw (untyped) buffers.
constexpr int kBufferWord3 = 0x00020000;
constexpr int kLdsRow = kWgBN + 32;          // row stride 576 B: rows fall 64 B apart in the banks
constexpr int kStage = kWgBK * kLdsRow;      // elements per operand and stage
constexpr int kChunks = kWgBK * kWgBN / 8 / kWgThreads;  // 16-byte chunks per lane, operand and stage
static_assert(kWgBM == kWgBN, "square tiles: one load pattern serves both operands");
static_assert(kChunks == 8, "load pattern");

// fp32 -> bf16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t to_bf16(float v) {
  const uint32_t u = __float_as_uint(v);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_val(uint32_t b) { return __uint_as_float(b << 16); }

__device__ __forceinline__ bf16x8 frag(const uint16_t* p0, const uint16_t* p1) {
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p1);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

__global__ __launch_bounds__(kWgThreads) void k5_wgrad(const WgBatch batch) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][kStage];  // [stage][x, dy]
  __shared__ float red[kWgThreads / 64];

  // Workgroup -> tile: workgroups w, w+8, ... run on one XCD, so give each
  // XCD a contiguous run of the tile order (over all problems of the batch);
  // inside a problem the order walks groups of 8 tile rows column by column,
  // so that the tiles an XCD holds at once share their dy and x panels in
  // its L2.
  const int G = batch.total_tiles;
  const int w = blockIdx.x;
  const int xcd = w % kNumXcd, q = G / kNumXcd, r = G % kNumXcd;
  int v = xcd * q + (xcd < r ? xcd : r) + w / kNumXcd;
  int pi = 0;
  while (pi + 1 < batch.num && v >= batch.p[pi + 1].tile_begin) ++pi;
  const WgProblem& P = batch.p[pi];
  v -= P.tile_begin;
  const uint16_t* __restrict__ dy = P.dy;
  const uint16_t* __restrict__ x = P.x;
  uint16_t* __restrict__ dw = P.dw;
  const int64_t K = P.K;
  const int M = P.M, N = P.N, tiles_m = P.tiles_m, tiles_n = P.tiles_n;
  const int per_group = kWgGroupRows * tiles_n;
  const int first_m = (v / per_group) * kWgGroupRows;
  const int rows = tiles_m - first_m < kWgGroupRows ? tiles_m - first_m : kWgGroupRows;
  const int tm = first_m + (v % per_group) % rows;
  const int tn = (v % per_group) / rows;
  const int m0 = tm * kWgBM, n0 = tn * kWgBN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;  // this wave's 128x128 quarter

  // Global -> LDS: lane tid moves 16-byte chunk (row tid/32 + 8c, column
  // 8*(tid%32)) of each operand tile, c = 0..7, with buffer loads whose
  // resource covers the rows of the current K step: rows past K and columns
  // past M or N (whose offset is pushed past the resource) read as zero in
  // hardware, so every load is issued unconditionally (M, N multiples of 8:
  // a chunk is all in or all out).
  const int lrow = tid >> 5, lcol = (tid & 31) * 8;
  const uint32_t kOut = 0x80000000u;  // beyond any resource of this kernel
  const uint32_t xo = n0 + lcol < N ? uint32_t((lrow * N + n0 + lcol) * 2) : kOut;
  const uint32_t yo = m0 + lcol < M ? uint32_t((lrow * M + m0 + lcol) * 2) : kOut;
  u32x4 rx[kChunks], ry[kChunks];
  auto gload = [&](int64_t k0) {
    const int rows = K - k0 < kWgBK ? int(K - k0) : kWgBK;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(x + k0 * N), 0, rows * N * 2, kBufferWord3);
    const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(dy + k0 * M), 0, rows * M * 2, kBufferWord3);
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      rx[c] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, xo + uint32_t(c * 16 * N), 0, 0));
      ry[c] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(yr, yo + uint32_t(c * 16 * M), 0, 0));
    }
  };
  auto lstore = [&](int st) {
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      *(u32x4*)&lds[st][0][(lrow + 8 * c) * kLdsRow + lcol] = rx[c];
      *(u32x4*)&lds[st][1][(lrow + 8 * c) * kLdsRow + lcol] = ry[c];
    }
  };

  // Fragment addressing for ds_read_b64_tr_b16: within each 16-lane group the
  // read hands lane i column i of the 4x16 block that the group's 8-byte
  // chunks form (chunk of lane 4j + c = row j, columns 4c..4c+3).  Lane l
  // then holds feature l%32 of a 32-wide block and k = 8*(l/32) + 4h + j for
  // the two reads h = 0, 1: the same k order for both operands.
  const int f_row = 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int f_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

  const int64_t nk = (K + kWgBK - 1) / kWgBK;  // 0 for an empty batch: dw = 0
  if (nk > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int64_t s = 0; s < nk; ++s) {
    const int st = int(s & 1);
    if (s + 1 < nk) gload((s + 1) * kWgBK);
    const uint16_t* lx = &lds[st][0][f_row * kLdsRow + wn * 128 + f_col];
    const uint16_t* ly = &lds[st][1][f_row * kLdsRow + wm * 128 + f_col];
#pragma unroll
    for (int kk = 0; kk < kWgBK / 16; ++kk) {
      bf16x8 fx[4], fy[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int o = kk * 16 * kLdsRow + 32 * b;
        fx[b] = frag(lx + o, lx + o + 4 * kLdsRow);
        fy[b] = frag(ly + o, ly + o + 4 * kLdsRow);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fx[j], fy[i], acc[i][j], 0, 0, 0);
    }
    if (s + 1 < nk) lstore(st ^ 1);
    __syncthreads();
  }

  // Epilogue: accumulator register r of block (i, j) holds output row
  // m = m0 + 128*wm + 32*i + lane%32 and column
  // n = n0 + 128*wn + 32*j + 8*(r/4) + 4*(lane/32) + r%4.
  float ss = 0.0f;
  const int m_lane = m0 + wm * 128 + (lane & 31);
  const int n_lane = n0 + wn * 128 + 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m_lane + 32 * i;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n_lane + 32 * j + 8 * g;
        const uint32_t b0 = to_bf16(acc[i][j][4 * g + 0]);
        const uint32_t b1 = to_bf16(acc[i][j][4 * g + 1]);
        const uint32_t b2 = to_bf16(acc[i][j][4 * g + 2]);
        const uint32_t b3 = to_bf16(acc[i][j][4 * g + 3]);
        if (m < M && n < N) {
          const float q0 = bf16_val(b0), q1 = bf16_val(b1), q2 = bf16_val(b2),
                      q3 = bf16_val(b3);
          ss = fmaf(q0, q0, ss);
          ss = fmaf(q1, q1, ss);
          ss = fmaf(q2, q2, ss);
          ss = fmaf(q3, q3, ss);
          *(g_vec2*)(dw + int64_t(m) * N + n) = u32x2{b0 | (b1 << 16), b2 | (b3 << 16)};
        }
      }
    }
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) ss += __shfl_xor(ss, d, 64);
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  if (tid == 0) P.tile_ss[tm * tiles_n + tn] = ((red[0] + red[1]) + red[2]) + red[3];
}

}  // namespace

int64_t wgrad_tiles(int32_t M, int32_t N) {
  return int64_t((M + kWgBM - 1) / kWgBM) * int64_t((N + kWgBN - 1) / kWgBN);
}

hipError_t launch_wgrad(const WgBatch& batch, hipStream_t s) {
  if (batch.total_tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(k5_wgrad, dim3(unsigned(batch.total_tiles)), dim3(kWgThreads), 0, s, batch);
  return hipGetLastError();
}

}  // namespace gnmr
