// Internal launch interface between the C ABI (uf_api.cpp) and the gfx950
// kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "uf.h"

namespace uf {

// Bytes of one page: K, then V^T, T*D bf16 each.  128-token pages keep both
// in blocks of 64 columns (K: [2][T][64] dimension halves, V^T: [2][D][64]
// key halves); 64-token pages hold K [T][D] and V^T [D][T].
__host__ __device__ inline size_t page_bytes(int T, int D) { return size_t(4) * size_t(T) * size_t(D); }

// Column of key r inside its group of 16 in a V^T page row: bits 2 and 3
// swapped.  The map is its own inverse.
__host__ __device__ inline int swap23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Valid rows of the tiles of a chunk: the last tile holds `tail` rows, unless
// the window has block geometry, whose per-block counts are tabulated.
struct TileValid {
  int32_t blocked;                 // 0: raster tiles
  int32_t nbh, nbw;                // block rows and columns of the grid (blocked)
  int32_t local_half;              // M_local half-width in blocks, -1: no local mask
  // valid rows of tile t (blocked): byte t % 4 of word t / 4, so that a
  // uniform index reads the kernel arguments with one scalar load (a byte
  // read would be a vector load, and the wait for it a wait for every copy
  // in flight)
  uint32_t count4[UF_MAX_BLOCKS / 4];
};
__host__ __device__ inline int tile_valid(const TileValid& v, int t, int NT, int tail, int T) {
  return v.blocked ? int((v.count4[t >> 2] >> (8 * (t & 3))) & 0xffu) : ((t == NT - 1) ? tail : T);
}
// M_local between query tile i and key tile t (block indices of one chunk).
__host__ __device__ inline bool tile_local(const TileValid& v, int i, int t) {
  if (v.local_half < 0) return true;
  const int dh = (i / v.nbw) % v.nbh - (t / v.nbw) % v.nbh;
  const int dw = i % v.nbw - t % v.nbw;
  return (dh <= v.local_half && -dh <= v.local_half) && (dw <= v.local_half && -dw <= v.local_half);
}

struct AppendArgs {
  const uint16_t* k;      // [B, L, H, D]
  const uint16_t* v;      // [B, L, H, D]
  uint8_t* pool;
  float* kmean;           // pooled keys of the pool: [slots][B][H][NT][D]
  int64_t slot;
  int32_t B, H, L, T, NT, tail;
  uint16_t pad;           // bf16 bits written into padding rows
  TileValid tv;
};
hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream);

struct ListArgs {
  uint8_t* lists;
  size_t idx_offset, mask_offset;
  int32_t rows;           // B*H*NT
  int32_t H, NT, nk, nk_cap, mask_words;
  uint64_t seed;
  uint64_t thr;           // 0 .. 2^32
  int32_t keep_sink, keep_current;
  int64_t cur_seq;
  int64_t seq[UF_MAX_CHUNKS];   // per logical position
  int32_t sink[UF_MAX_CHUNKS];  // 1 if logical position holds the pinned chunk
  TileValid tv;
};
hipError_t launch_tile_lists(const ListArgs& a, hipStream_t stream);

// Top-k lists: one workgroup per (b, h, group of G query tiles).
struct TopkArgs {
  const uint16_t* q;      // [B, L, H, D]
  const float* kmean;     // pooled keys: [slots][B][H][NT][D]
  uint8_t* lists;
  size_t idx_offset, mask_offset, scratch_offset;   // scratch: pooled queries [B][H][NT][D]
  int32_t B, H, L, T, NT, tail, nk, nk_cap, mask_words;
  int32_t G;              // query tiles per workgroup
  int32_t cand_lo, cand_hi;   // ranked logical tiles [cand_lo, cand_hi)
  int32_t budget;
  int32_t slot_of[UF_MAX_CHUNKS];
  TileValid tv;
};
constexpr int kTopkMaxCandidates = 16384;   // G * candidates per workgroup
hipError_t launch_topk_lists(const TopkArgs& a, size_t lds_bytes, hipStream_t stream);

struct AttnArgs {
  const uint16_t* q;      // [B, L, H, D]
  uint16_t* o;            // [B, L, H, D]
  float* lse;             // [B, H, L] or null
  const uint8_t* pool;
  const int32_t* counts;  // [rows]
  const int32_t* idx;     // [rows][nk_cap]
  int32_t B, H, L, T, NT, tail, nk, nk_cap;
  uint64_t nt_div;        // (2^64 - 1) / NT: j / NT == ((j + 1) * nt_div) >> 64 for 0 <= j < 2^31
  float scale;            // softmax scale
  float scale_log2;       // scale * log2(e)
  int32_t split;          // list slices per split row (split-KV), 1 = whole rows
  int32_t split_from;     // split-KV: rows before this one run whole (0: every row is split)
  float* work;            // split-KV partials of the split rows R = rows - split_from:
                          // O [R*split][T][D], then (m, l) [R*split][T]
  int32_t slot_of[UF_MAX_CHUNKS];  // slot of each logical position
  TileValid tv;
};

// Block-order permutation of [B, tokens, H, 128] bf16 rows.
struct PermuteArgs {
  const uint16_t* src;
  uint16_t* dst;
  int32_t B, H, frames, gh, gw, bt, bh, bw, nbh, nbw, tokens, padded, inverse;
};
hipError_t launch_block_permute(const PermuteArgs& a, hipStream_t stream);
hipError_t launch_attn_fwd_t64(const AttnArgs& a, hipStream_t stream);
hipError_t launch_attn_fwd_t128_tri(const AttnArgs& a, hipStream_t stream);
hipError_t launch_attn_fwd_t128_tri_split(const AttnArgs& a, hipStream_t stream);
hipError_t launch_attn_fwd_t64_split(const AttnArgs& a, hipStream_t stream);
// combines the split-KV partials in a.work into O and LSE (rows split_from ..)
hipError_t launch_attn_split_merge(const AttnArgs& a, hipStream_t stream);

inline hipError_t launch_attn_fwd(const AttnArgs& a, hipStream_t stream) {
  return a.T == 128 ? launch_attn_fwd_t128_tri(a, stream) : launch_attn_fwd_t64(a, stream);
}
// split-KV launch (a.split, a.split_from, a.work set) and its merge
inline hipError_t launch_attn_fwd_split(const AttnArgs& a, hipStream_t stream) {
  return a.T == 128 ? launch_attn_fwd_t128_tri_split(a, stream) : launch_attn_fwd_t64_split(a, stream);
}

}  // namespace uf
