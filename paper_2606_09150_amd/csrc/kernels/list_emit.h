// Output stage shared by the list builders: one workgroup of 256 lanes writes
// the list row of one (b, h, query tile) from a keep predicate over logical
// key tiles 0 .. nk_cap-1 (false at and beyond nk).  Each pass decides 256
// consecutive tiles; a wave ballot gives two 32-bit mask words per wave and a
// prefix over the four wave counts places the kept indices in ascending
// order; the tail of the row is padded with -1.
#pragma once

#include "../launch.h"

namespace uf {
namespace lists {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

// `wave_count` is a __shared__ int[kWaves] of the calling kernel.  Every lane
// of the workgroup must call this (it contains barriers).
template <class Keep>
__device__ void emit_row(Keep keep_of, int nk_cap, int mask_words, int32_t* count, int32_t* idx,
                         uint32_t* mask, int* wave_count) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int base = 0;
  for (int j0 = 0; j0 < nk_cap; j0 += kThreads) {
    const int j = j0 + threadIdx.x;
    const bool keep = (j < nk_cap) && keep_of(j);
    const uint64_t ballot = __ballot(keep);
    const int w0 = (j0 + wave * 64) >> 5;
    if (lane == 0 && w0 < mask_words) mask[w0] = uint32_t(ballot);
    if (lane == 0 && w0 + 1 < mask_words) mask[w0 + 1] = uint32_t(ballot >> 32);
    if (lane == 0) wave_count[wave] = __popcll(ballot);
    __syncthreads();
    int off = base, total = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      off += (w < wave) ? wave_count[w] : 0;
      total += wave_count[w];
    }
    if (keep) idx[off + __popcll(ballot & ((1ull << lane) - 1ull))] = j;
    __syncthreads();
    base += total;
  }
  for (int j = base + threadIdx.x; j < nk_cap; j += kThreads) idx[j] = -1;
  if (threadIdx.x == 0) *count = base;
}

}  // namespace lists
}  // namespace uf
