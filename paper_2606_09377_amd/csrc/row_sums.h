// Constant-term row sums of the MFMA epilogues, shared by the GEMM and the transposed
// convolution.
#pragma once

#include <hip/hip_runtime.h>

namespace vcr {

// A half-wave (32 lanes, one column each) holds the constant terms of 16 rows, one value per
// row and lane (rp[v]).  Returns the sum over the 32 lanes of row (r32 >> 1) & 15.  This is
// the butterfly x += shfl_xor(x, 16), (x, 8), (x, 4), (x, 2), (x, 1) of every row, done as a
// reduce-scatter: at each of the first four levels a lane keeps half of its rows and sends the
// other half to its partner, so 16 exchanges replace 80.  Each level adds the same two
// operands in the same order as the per-row butterfly (own value first), and a pairwise sum is
// the same either way round, so every lane holding a row ends with the bits that the per-row
// butterfly leaves in every lane.
__device__ __forceinline__ float half_wave_row_sums(const float (&rp)[16], int r32) {
  const bool b4 = r32 & 16, b3 = r32 & 8, b2 = r32 & 4, b1 = r32 & 2;
  float v8[8], v4[4], v2[2];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float send = b4 ? rp[j] : rp[j + 8], keep = b4 ? rp[j + 8] : rp[j];
    v8[j] = keep + __shfl_xor(send, 16);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float send = b3 ? v8[j] : v8[j + 4], keep = b3 ? v8[j + 4] : v8[j];
    v4[j] = keep + __shfl_xor(send, 8);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float send = b2 ? v4[j] : v4[j + 2], keep = b2 ? v4[j + 2] : v4[j];
    v2[j] = keep + __shfl_xor(send, 4);
  }
  const float send = b1 ? v2[0] : v2[1], keep = b1 ? v2[1] : v2[0];
  float x = keep + __shfl_xor(send, 2);
  x += __shfl_xor(x, 1);
  return x;
}

// Eight values per lane summed over the 64 lanes of a wave, as the same kind of
// reduce-scatter over the butterfly x += shfl_xor(x, 32), (x, 16), ..., (x, 1): returns the
// sum of value (lane >> 3) & 7, with the per-value butterfly's bits.
__device__ __forceinline__ float wave_sums8(const float (&v)[8], int lane) {
  const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
  float v4[4], v2[2];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float send = b5 ? v[j] : v[j + 4], keep = b5 ? v[j + 4] : v[j];
    v4[j] = keep + __shfl_xor(send, 32);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float send = b4 ? v4[j] : v4[j + 2], keep = b4 ? v4[j + 2] : v4[j];
    v2[j] = keep + __shfl_xor(send, 16);
  }
  const float send = b3 ? v2[0] : v2[1], keep = b3 ? v2[1] : v2[0];
  float x = keep + __shfl_xor(send, 8);
  x += __shfl_xor(x, 4);
  x += __shfl_xor(x, 2);
  x += __shfl_xor(x, 1);
  return x;
}

}  // namespace vcr
