// K5, the gradient pass fused into its producer for CDNA4 (gfx950): the
// weight-gradient GEMM of a linear layer with the sum of squares that the
// controller needs computed in its epilogue, so that the gradient is never
// read back from HBM for its norm (the norm is the only per-unit quantity
// the controller takes from the gradient, Sec. 3.3 and Alg. 1; it is cheap
// to compute from what the producer already holds, Sec. 3.1).
//
//   dw[o][i] = bf16_rne( sum_t dy[t][o] * x[t][i] )   fp32 accumulation
//   (accumulating problems: bf16_rne( fp32(dw_old[o][i] + that sum) ))
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
// 128x128 (4x4 v_mfma_f32_32x32x16_bf16 blocks each), K steps of 64 split
// into four slots of 16 (one matrix-core instruction per block and slot).
// Two LDS buffers and one set of staging registers form the pipeline:
// during step s the matrix cores work on buffer s%2, the staged operands of
// step s+1 go to the other buffer while the global loads of step s+2 refill
// the staging registers, so every global load has a whole step to land.
// The fragments of slot k+1 are read from LDS while slot k's matrix-core
// instructions run (two fragment register sets), and the workgroup meets at
// one barrier per step, placed before the last slot's matrix-core work so
// that the reads of the next buffer overlap it.  x is the matrix cores' A
// operand, so the four accumulator rows a lane holds per group are four
// consecutive output columns, 8 contiguous bytes once rounded.  Overwritten
// tiles that lie wholly inside dw pass through LDS and leave as full rows;
// the others store each lane's 8 bytes directly.

#include "gnmr_internal.h"

namespace gnmr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) u32x2 g_vec2;
typedef __attribute__((address_space(1))) u32x4 g_vec4;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Buffer resource word 3 for gfx9-family raw (untyped) buffers.
constexpr int kBufferWord3 = 0x00020000;
constexpr int kLdsRow = kWgBN + 32;          // row stride 576 B: rows fall 64 B apart in the banks
constexpr int kStage = kWgBK * kLdsRow;      // elements per operand and stage
constexpr int kChunks = kWgBK * kWgBN / 8 / kWgThreads;  // 16-byte chunks per lane, operand and stage
static_assert(kWgBM == kWgBN, "square tiles: one load pattern serves both operands");
static_assert(kChunks == 8, "load pattern");
static_assert(kWgBK == 64, "four slots of 16 per K step");
// sched_group_barrier instruction classes
constexpr int kSchedMfma = 0x008;
constexpr int kSchedVmemRead = 0x020;
constexpr int kSchedDsRead = 0x100;
constexpr int kSchedDsWrite = 0x200;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values to packed bf16 (lo in the low half), round to nearest
// even, a NaN to a quiet NaN with its payload kept: one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ float bf16_val(uint32_t b) { return __uint_as_float(b << 16); }

__device__ __forceinline__ bf16x8 frag(const uint16_t* p0, const uint16_t* p1) {
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p0);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p1);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// kAcc: every problem of the batch accumulates into its stored dw (true) or
// overwrites it (false); a batch of both kinds takes one launch of each.
template <bool kAcc>
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
  // resource covers the rows of one K step: rows past K and columns past M
  // or N (whose offset is pushed past the resource) read as zero in
  // hardware, so every load is issued unconditionally (M, N multiples of 8:
  // a chunk is all in or all out).  Steps past the end get an empty
  // resource: their loads read zeros without touching memory, and the
  // buffers they fill are never read, which keeps the loop body free of
  // branches.
  const int lrow = tid >> 5, lcol = (tid & 31) * 8;
  const uint32_t kOut = 0x80000000u;  // beyond any resource of this kernel
  const uint32_t xo = n0 + lcol < N ? uint32_t((lrow * N + n0 + lcol) * 2) : kOut;
  const uint32_t yo = m0 + lcol < M ? uint32_t((lrow * M + m0 + lcol) * 2) : kOut;
  u32x4 rx[kChunks], ry[kChunks];
  __amdgpu_buffer_rsrc_t xr, yr;
  auto rsrc = [&](int64_t k0) {
    const int64_t kb = k0 < K ? k0 : 0;
    const int rws = k0 >= K ? 0 : (K - k0 < kWgBK ? int(K - k0) : kWgBK);
    xr = __builtin_amdgcn_make_buffer_rsrc((void*)(x + kb * N), 0, rws * N * 2, kBufferWord3);
    yr = __builtin_amdgcn_make_buffer_rsrc((void*)(dy + kb * M), 0, rws * M * 2, kBufferWord3);
  };
  auto gload = [&](int h) {  // chunks 4h .. 4h+3 of both operands
#pragma unroll
    for (int c = 4 * h; c < 4 * h + 4; ++c) {
      rx[c] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, xo + uint32_t(c * 16 * N), 0, 0));
      ry[c] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(yr, yo + uint32_t(c * 16 * M), 0, 0));
    }
  };
  auto lstore = [&](int buf, int h) {
#pragma unroll
    for (int c = 4 * h; c < 4 * h + 4; ++c) {
      *(u32x4*)&lds[buf][0][(lrow + 8 * c) * kLdsRow + lcol] = rx[c];
      *(u32x4*)&lds[buf][1][(lrow + 8 * c) * kLdsRow + lcol] = ry[c];
    }
  };

  // Fragment addressing for ds_read_b64_tr_b16: within each 16-lane group the
  // read hands lane i column i of the 4x16 block that the group's 8-byte
  // chunks form (chunk of lane 4j + c = row j, columns 4c..4c+3).  Lane l
  // then holds feature l%32 of a 32-wide block and k = 8*(l/32) + 4h + j for
  // the two reads h = 0, 1: the same k order for both operands.
  const int f_row = 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int f_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  bf16x8 fx[2][4], fy[2][4];  // [register set][block]
  auto rfrag = [&](int set, int buf, int kk) {
    const uint16_t* lx = &lds[buf][0][f_row * kLdsRow + wn * 128 + f_col];
    const uint16_t* ly = &lds[buf][1][f_row * kLdsRow + wm * 128 + f_col];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int o = kk * 16 * kLdsRow + 32 * b;
      fx[set][b] = frag(lx + o, lx + o + 4 * kLdsRow);
      fy[set][b] = frag(ly + o, ly + o + 4 * kLdsRow);
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
  auto mfma = [&](int set) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] =
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(fx[set][j], fy[set][i], acc[i][j], 0, 0, 0);
  };
  // Instruction order inside a slot (scheduling hints only): each
  // matrix-core instruction is followed by two fragment reads for the next
  // slot, then, in slots 0 and 1, by one LDS store and one global load.
  auto order_reads = [] {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
    }
  };
  auto order_stores = [] {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedDsWrite, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedVmemRead, 1, 0);
    }
  };

  // 0 steps for an empty batch: dw = 0.  Prologue: step 0 in buffer 0,
  // step 1 in the staging registers, the first slot's fragments read.
  const int64_t nk = (K + kWgBK - 1) / kWgBK;
  rsrc(0);
  gload(0);
  gload(1);
  lstore(0, 0);
  lstore(0, 1);
  rsrc(kWgBK);
  gload(0);
  gload(1);
  __syncthreads();
  rfrag(0, 0, 0);
  for (int64_t s = 0; s < nk; ++s) {
    const int buf = int(s & 1);
    // slot 0: stage half of step s+1, load half of step s+2
    rfrag(1, buf, 1);
    lstore(buf ^ 1, 0);
    rsrc((s + 2) * kWgBK);
    gload(0);
    mfma(0);
    order_reads();
    order_stores();
    // slot 1: the other halves
    rfrag(0, buf, 2);
    lstore(buf ^ 1, 1);
    gload(1);
    mfma(1);
    order_reads();
    order_stores();
    // slot 2
    rfrag(1, buf, 3);
    mfma(0);
    order_reads();
    __builtin_amdgcn_sched_group_barrier(kSchedMfma, 8, 0);
    // slot 3: every wave has stored its part of step s+1 and read its last
    // fragments of buffer s%2 (the barrier waits for both), so buffer
    // (s+1)%2 is complete and buffer s%2 free for step s+2
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    rfrag(0, buf ^ 1, 0);
    mfma(1);
    order_reads();
    __builtin_amdgcn_sched_group_barrier(kSchedMfma, 8, 0);
  }

  // Epilogue: accumulator register r of block (i, j) holds output row
  // m = m0 + 128*wm + 32*i + lane%32 and column
  // n = n0 + 128*wn + 32*j + 8*(r/4) + 4*(lane/32) + r%4.  When the problem
  // accumulates, the stored gradient is first widened and added in fp32 (one
  // rounding), then the sum is rounded to bf16 once.
  float ss = 0.0f;
  const int m_lane = m0 + wm * 128 + (lane & 31);
  const int n_lane = n0 + wn * 128 + 4 * (lane >> 5);
  // Accumulating: the stored tile is first copied into the LDS buffers (free
  // once the loop is done) by direct-to-LDS 16-byte loads, which need no
  // registers: each wavefront instruction fills two rows of 512 B, and chunk
  // c of row r sits in slot c ^ (r % 32) of its row, so that the epilogue's
  // reads of 32 consecutive rows at one column spread over the banks.  Loads
  // of rows or columns outside dw read dw[0] instead (never used).
  uint16_t* const old_tile = &lds[0][0][0];
  static_assert(kWgBM * kWgBN <= 2 * 2 * kStage, "the stored tile fits in the LDS buffers");
  auto stage_old = [&]() {
    __syncthreads();  // every wave is done with the operand buffers
    const int row_in_pair = lane >> 5, slot = lane & 31;
#pragma unroll 1
    for (int q = 0; q < kWgBM / 2 / 4; ++q) {  // 32 row pairs per wave
      const int row = (wave * (kWgBM / 8) + q) * 2 + row_in_pair;
      const int m = m0 + row, n = n0 + 8 * (slot ^ (row & 31));
      const uint16_t* src = (m < M && n < N) ? dw + int64_t(m) * N + n : dw;
      __builtin_amdgcn_global_load_lds(
          (const void*)src,
          (__attribute__((address_space(3))) void*)(old_tile + (row & ~1) * kWgBN), 16, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };
  auto old_pair = [&](int m, int n) {  // the stored values at (m, n .. n+3)
    const int row = m - m0, c = (n - n0) >> 3, w = (n - n0) & 7;
    return *(const u32x2*)&old_tile[row * kWgBN + 8 * (c ^ (row & 31)) + w];
  };
  // Rounds one group of four accumulator values (row m, columns n .. n+3)
  // and adds their squares to ss in a fixed order; returns them packed.
  auto round_group = [&](int i, int j, int g, int m, int n) {
    float v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1], v2 = acc[i][j][4 * g + 2],
          v3 = acc[i][j][4 * g + 3];
    if constexpr (kAcc) {
      const u32x2 old = old_pair(m, n);
      v0 += bf16_val(old.x & 0xFFFFu);
      v1 += bf16_val(old.x >> 16);
      v2 += bf16_val(old.y & 0xFFFFu);
      v3 += bf16_val(old.y >> 16);
    }
    const uint32_t p01 = pack_bf16(v0, v1), p23 = pack_bf16(v2, v3);
    const float q0 = __uint_as_float(p01 << 16), q1 = __uint_as_float(p01 & 0xFFFF0000u),
                q2 = __uint_as_float(p23 << 16), q3 = __uint_as_float(p23 & 0xFFFF0000u);
    ss = fmaf(q0, q0, ss);
    ss = fmaf(q1, q1, ss);
    ss = fmaf(q2, q2, ss);
    ss = fmaf(q3, q3, ss);
    return u32x2{p01, p23};
  };
  auto epilogue = [&]() {
    if constexpr (kAcc) stage_old();
    if (!kAcc && m0 + kWgBM <= M && n0 + kWgBN <= N) {
      // Overwriting a tile wholly inside dw (uniform): the rounded tile goes
      // to the free LDS buffers first, in the swizzled layout of the stored
      // tile, then leaves in full rows: each wavefront store covers two whole
      // 512-byte rows, where a lane's own accumulator layout would touch 32
      // rows with 16 bytes each.  (Accumulating, the same staging spills
      // registers and measured no faster, so those tiles store directly.)
      __syncthreads();  // every wave is done with the operand buffers
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          // one block at a time: its conversions and LDS accesses stay next
          // to their use, within the registers the accumulators leave free
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int m = m_lane + 32 * i, n = n_lane + 32 * j + 8 * g;
            const u32x2 v = round_group(i, j, g, m, n);
            const int row = m - m0, c = (n - n0) >> 3, w = (n - n0) & 7;
            *(u32x2*)&old_tile[row * kWgBN + 8 * (c ^ (row & 31)) + w] = v;
          }
        }
      }
      __syncthreads();
      const int c = tid & 31;
      int row = tid >> 5;
      uint16_t* out = dw + int64_t(m0 + row) * N + n0 + 8 * c;
#pragma unroll 4
      for (int p = 0; p < kWgBM * kWgBN / 8 / kWgThreads; ++p) {
        *(g_vec4*)out = *(const u32x4*)&old_tile[row * kWgBN + 8 * (c ^ (row & 31))];
        row += kWgThreads / 32;
        out += int64_t(kWgThreads / 32) * N;
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m_lane + 32 * i;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = n_lane + 32 * j + 8 * g;
          if (m < M && n < N) *(g_vec2*)(dw + int64_t(m) * N + n) = round_group(i, j, g, m, n);
        }
      }
    }
  };
  epilogue();
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
  // one launch per epilogue kind: the problems that overwrite dw, then those
  // that accumulate into it, each launch with its own tile order
  for (const int acc : {0, 1}) {
    WgBatch b{};
    for (int i = 0; i < batch.num; ++i) {
      if ((batch.p[i].accumulate != 0) != (acc != 0)) continue;
      WgProblem P = batch.p[i];
      P.tile_begin = b.total_tiles;
      b.total_tiles += P.tiles_m * P.tiles_n;
      b.p[b.num++] = P;
    }
    if (b.total_tiles == 0) continue;
    if (acc)
      hipLaunchKernelGGL(k5_wgrad<true>, dim3(unsigned(b.total_tiles)), dim3(kWgThreads), 0, s, b);
    else
      hipLaunchKernelGGL(k5_wgrad<false>, dim3(unsigned(b.total_tiles)), dim3(kWgThreads), 0, s,
                         b);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace gnmr
