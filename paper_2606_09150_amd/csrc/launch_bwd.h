// Launch interface of the attention backward (internal to libuf.so).
#pragma once

#include "launch.h"

namespace uf {

// Backward of the attention.  The workspace holds, per query tile (b, h, i),
// the Q and dO rows (zero past the chunk end), then -LSE/scale (-inf past the
// chunk end) and -delta = -<dO, O> per query.
constexpr size_t kBwdQTile = 2 * 32768 + 1024;
constexpr int kBwdMaxQTiles = 2048;   // query tiles per chunk the backward handles
struct BwdArgs {
  const uint16_t* q;      // [B, L, H, D]
  const uint16_t* o;      // [B, L, H, D]
  const uint16_t* dout;   // [B, L, H, D]
  const float* lse;       // [B, H, L]
  const uint8_t* pool;
  const int32_t* counts;  // lists
  const int32_t* idx;
  const uint32_t* mask;
  float* dq;              // [B, L, H, D]
  float* dk;              // [n_live][B, L, H, D]
  float* dv;              // [n_live][B, L, H, D]
  uint8_t* work;
  int32_t B, H, L, T, NT, tail, nk, nk_cap, mask_words, n_live;
  float scale, scale_log2;
  int32_t slot_of[UF_MAX_CHUNKS];
  TileValid tv;
};
hipError_t launch_attn_bwd(const BwdArgs& a, hipStream_t stream);
// The same launches with the query-tile records in the library's own device
// scratch (kBwdScratchBytes per GPU) instead of a.work; needs
// B*H*NT*kBwdQTile <= kBwdScratchBytes (hipErrorInvalidValue otherwise).
// Allocates nothing; calls that overlap on one GPU race.
constexpr size_t kBwdScratchBytes = UF_BWD_SCRATCH_BYTES;
hipError_t launch_attn_bwd_noalloc(BwdArgs a, hipStream_t stream);

}  // namespace uf
