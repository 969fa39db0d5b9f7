// 128 x 128 output tile of C[i][j] = sum_k P[i][k] * Q[j][k] on bf16 MFMA.
//
// Both operands are row-major with the contraction index contiguous, so the
// same core serves the similarity (Gram) tiles, where P and Q are gathered
// token rows, and the FFN tiles, where P holds weight rows ([out, in]
// layout) and Q gathered token rows.
//
// 256 threads = 4 waves in a 2 x 2 grid, each wave owning a 64 x 64 sub-tile
// made of 4 x 4 MFMA 16x16x32 blocks.  K advances 64 at a time through
// double-buffered LDS (rows padded by 8 elements against bank conflicts);
// the next K slice is fetched into registers while the current one is
// multiplied.
//
// Result layout: acc[i][j][r] holds
//   P row  64*(wave/2) + 16*i + 4*(lane/16) + r
//   Q row  64*(wave%2) + 16*j + lane%16
#pragma once

#include "luffy_common.h"

namespace luffy {

constexpr int kTile = 128;
constexpr int kTileK = 64;
constexpr int kLdsStride = kTileK + 8;                 // bf16 elements per LDS row
constexpr int kTileLdsElems = 4 * kTile * kLdsStride;  // P and Q, double-buffered

// Rows this thread loads: (tid / 8) + 32 * q, q = 0..3, columns (tid % 8) * 8.
__device__ __forceinline__ void gemm_tile_bf16(const uint16_t* const prow[4],
                                               const uint16_t* const qrow[4], int K,
                                               uint16_t* __restrict__ lds,
                                               f32x4 (&acc)[4][4]) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int col = (tid & 7) * 8;
  const int lrow = tid >> 3;
  // buffer b of P at lds + b*BUF, of Q at lds + (2+b)*BUF
  constexpr int BUF = kTile * kLdsStride;

  uint4 pr[4], qr[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    pr[q] = *reinterpret_cast<const uint4*>(prow[q] + col);
    qr[q] = *reinterpret_cast<const uint4*>(qrow[q] + col);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    *reinterpret_cast<uint4*>(lds + (lrow + 32 * q) * kLdsStride + col) = pr[q];
    *reinterpret_cast<uint4*>(lds + 2 * BUF + (lrow + 32 * q) * kLdsStride + col) = qr[q];
  }
  __syncthreads();

  const int nk = K / kTileK;
  const int arow = (lane & 15) * kLdsStride + 8 * (lane >> 4);
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    // the last iteration re-reads its own slice, so no branch guards the
    // register prefetch (keeps pr/qr in registers)
    const int k0 = (kt + 1 < nk ? kt + 1 : kt) * kTileK + col;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      pr[q] = *reinterpret_cast<const uint4*>(prow[q] + k0);
      qr[q] = *reinterpret_cast<const uint4*>(qrow[q] + k0);
    }
    const uint16_t* P = lds + cur * BUF + (64 * wm) * kLdsStride + arow;
    const uint16_t* Q = lds + (2 + cur) * BUF + (64 * wn) * kLdsStride + arow;
#pragma unroll
    for (int kk = 0; kk < kTileK; kk += 32) {
      bf16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(P + 16 * i * kLdsStride + kk);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(Q + 16 * j * kLdsStride + kk);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(a[i], b[j], acc[i][j]);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *reinterpret_cast<uint4*>(lds + (cur ^ 1) * BUF + (lrow + 32 * q) * kLdsStride + col) = pr[q];
      *reinterpret_cast<uint4*>(lds + (3 - cur) * BUF + (lrow + 32 * q) * kLdsStride + col) = qr[q];
    }
    __syncthreads();
  }
}

__device__ __forceinline__ void zero_acc(f32x4 (&acc)[4][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
}

}  // namespace luffy
