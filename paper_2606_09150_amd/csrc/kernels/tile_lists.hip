// tile_lists: per (b, h, query tile) keep lists of key tiles.
//
// Realises the block mask of Eq. 4 (Sec. 2.3.1): the temporal causal mask
// (the current chunk sees the window's earlier chunks and itself) intersected
// with a keep set.  The keep set here is the seeded Bernoulli stand-in for the
// content-adaptive top-k: pinned and current chunks always kept, every other
// key tile kept iff the upper 32 bits of a SplitMix64 chain over
// (b, h, seq(current), i, seq(chunk), t) fall below floor(p * 2^32).
//
// One workgroup of 256 lanes per list row; the row is written by the shared
// output stage (list_emit.h).  Integer-only, so the lists are bit-exact.
#include "list_emit.h"

namespace uf {
namespace {

using lists::kThreads;
using lists::kWaves;

// One SplitMix64 step (Steele, Lea, Flood, OOPSLA 2014): golden-ratio
// increment, then the 64-bit finaliser.
__device__ inline uint64_t splitmix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ __launch_bounds__(kThreads) void tile_lists_kernel(ListArgs a) {
  __shared__ int wave_count[kWaves];

  const int row = blockIdx.x;
  const int i = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  uint64_t x = a.seed;
  x = splitmix64(x ^ uint64_t(b));
  x = splitmix64(x ^ uint64_t(h));
  x = splitmix64(x ^ uint64_t(a.cur_seq));
  x = splitmix64(x ^ uint64_t(i));

  int32_t* counts = reinterpret_cast<int32_t*>(a.lists);
  int32_t* idx = reinterpret_cast<int32_t*>(a.lists + a.idx_offset) + size_t(row) * a.nk_cap;
  uint32_t* mask = reinterpret_cast<uint32_t*>(a.lists + a.mask_offset) + size_t(row) * a.mask_words;

  auto keep_of = [&](int j) {
    if (j >= a.nk) return false;
    const int pos = j / a.NT;
    const int t = j - pos * a.NT;
    if (!tile_local(a.tv, i, t)) return false;   // structural local window (block geometry)
    if ((a.sink[pos] && a.keep_sink) || (a.seq[pos] == a.cur_seq && a.keep_current)) return true;
    uint64_t y = splitmix64(x ^ uint64_t(a.seq[pos]));
    y = splitmix64(y ^ uint64_t(t));
    return (y >> 32) < a.thr;
  };
  lists::emit_row(keep_of, a.nk_cap, a.mask_words, counts + row, idx, mask, wave_count);
}

}  // namespace

hipError_t launch_tile_lists(const ListArgs& a, hipStream_t stream) {
  tile_lists_kernel<<<unsigned(a.rows), kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
