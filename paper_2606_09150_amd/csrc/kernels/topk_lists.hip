// topk_lists: per (b, h, query tile) keep lists by content-adaptive top-k.
//
// Realises the content-adaptive selection of Sec. 2.3.1 (b), Eq. 4: queries
// and keys are mean-pooled per tile, each (query tile, key tile) pair gets the
// dot product of the pooled vectors as its score, and every query tile keeps
// the `budget` best-scoring key tiles among the ranked candidates (the softmax
// and 1/sqrt(d) of Eq. 4 are monotone and do not change the ranking).  Tiles
// of the pinned and of the current chunk are kept without ranking when the
// rule asks for it; the lists are intersected with the temporal causal mask
// by construction (only the window's tiles exist).
//
// Arithmetic is IEEE float32 in a fixed order, so that the integer decision is
// reproducible: a pooled query is the sequential sum of the tile's valid rows
// divided once by their count (pooled keys come from the append kernel in the
// same form); a score adds the rounded products in order of d, with fused
// multiply-add disabled; scores compare through the unsigned key that orders
// float32 like the real line, equal keys going to the lower tile index.
//
// One workgroup of 256 lanes per (b, h, group of G query tiles): the G pooled
// queries sit in LDS, the pooled keys of the ranked candidates stream through
// LDS 32 tiles at a time and are shared by the G rows; a candidate is kept iff
// fewer than `budget` candidates of its row beat it (O(candidates^2) per row);
// each row is then written by the shared output stage.
#include "list_emit.h"

#pragma clang fp contract(off)

namespace uf {
namespace {

using lists::kThreads;
using lists::kWaves;
constexpr int kD = 128;
constexpr int kMaxG = 8;
constexpr int kStageTiles = 32;
constexpr int kStageStride = kD + 1;   // floats; the odd stride spreads LDS banks

__device__ inline float bf16_to_f32(uint16_t x) { return __uint_as_float(uint32_t(x) << 16); }

// Unsigned key that orders float32 values like the real line.
__device__ inline uint32_t order_key(float s) {
  const uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__global__ __launch_bounds__(kThreads) void topk_lists_kernel(TopkArgs a) {
  extern __shared__ uint32_t dyn[];
  __shared__ float qm[kMaxG][kD];
  __shared__ float kst[kStageTiles * kStageStride];
  __shared__ int wave_count[kWaves];

  const int nc = max(a.cand_hi - a.cand_lo, 0);   // ranked candidates of a row
  uint32_t* keys = dyn;                            // [G][nc]
  uint8_t* sel = reinterpret_cast<uint8_t*>(dyn + size_t(a.G) * nc);   // [G][nc]

  const int groups = (a.NT + a.G - 1) / a.G;
  const int grp = blockIdx.x % groups;
  const int bh = blockIdx.x / groups;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int i0 = grp * a.G;
  const int gn = min(a.G, a.NT - i0);
  const int tid = threadIdx.x;

  // 1. pooled queries: lane (half, d) sums column d of tiles half, half + 2, ...
  {
    const int d = tid & (kD - 1);
    const size_t rs = size_t(a.H) * kD;
    for (int g = tid >> 7; g < gn; g += 2) {
      const int i = i0 + g;
      const int nv = (i == a.NT - 1) ? a.tail : a.T;
      const uint16_t* qp = a.q + ((size_t(b) * a.L + size_t(i) * a.T) * a.H + h) * kD + d;
      float acc = 0.f;
      for (int r = 0; r < nv; ++r) acc += bf16_to_f32(qp[size_t(r) * rs]);
      qm[g][d] = acc / float(nv);
    }
  }

  // 2. scores of the ranked candidates
  const size_t slot_pages = size_t(a.B) * a.H * a.NT;
  const size_t head_page = size_t(bh) * a.NT;
  for (int m0 = 0; m0 < nc; m0 += kStageTiles) {
    __syncthreads();   // pooled queries written / previous stage consumed
    for (int e = tid; e < kStageTiles * kD; e += kThreads) {
      const int mt = e / kD;
      const int d = e - mt * kD;
      const int m = m0 + mt;
      float v = 0.f;
      if (m < nc) {
        const int j = a.cand_lo + m;
        const int pos = j / a.NT;
        const int t = j - pos * a.NT;
        v = a.kmean[(size_t(a.slot_of[pos]) * slot_pages + head_page + t) * kD + d];
      }
      kst[mt * kStageStride + d] = v;
    }
    __syncthreads();
    for (int p = tid; p < gn * kStageTiles; p += kThreads) {
      const int g = p / kStageTiles;
      const int mt = p - g * kStageTiles;
      const int m = m0 + mt;
      if (m < nc) {
        float acc = 0.f;
        for (int d = 0; d < kD; ++d) acc = acc + qm[g][d] * kst[mt * kStageStride + d];
        keys[size_t(g) * nc + m] = order_key(acc);
      }
    }
  }
  __syncthreads();

  // 3. selection: candidate m of row g is kept iff fewer than `budget`
  //    candidates of the row have a larger key, or an equal key and a lower index
  for (int p = tid; p < gn * nc; p += kThreads) {
    const int g = p / nc;
    const int m = p - g * nc;
    const uint32_t* row = keys + size_t(g) * nc;
    const uint32_t km = row[m];
    int beats = 0;
    for (int m2 = 0; m2 < nc; ++m2) {
      const uint32_t k2 = row[m2];
      beats += (k2 > km || (k2 == km && m2 < m)) ? 1 : 0;
    }
    sel[size_t(g) * nc + m] = beats < a.budget ? 1 : 0;
  }
  __syncthreads();

  // 4. the list rows
  int32_t* counts = reinterpret_cast<int32_t*>(a.lists);
  for (int g = 0; g < gn; ++g) {
    const int row = bh * a.NT + i0 + g;
    int32_t* idx = reinterpret_cast<int32_t*>(a.lists + a.idx_offset) + size_t(row) * a.nk_cap;
    uint32_t* mask = reinterpret_cast<uint32_t*>(a.lists + a.mask_offset) + size_t(row) * a.mask_words;
    const uint8_t* sg = sel + size_t(g) * nc;
    auto keep_of = [&](int j) {
      if (j >= a.nk) return false;
      if (j < a.cand_lo || j >= a.cand_hi) return true;   // forced: pinned or current chunk
      return sg[j - a.cand_lo] != 0;
    };
    lists::emit_row(keep_of, a.nk_cap, a.mask_words, counts + row, idx, mask, wave_count);
  }
}

}  // namespace

hipError_t launch_topk_lists(const TopkArgs& a, size_t lds_bytes, hipStream_t stream) {
  // the candidate keys and flags may take more than the default dynamic LDS
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(topk_lists_kernel),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     kTopkMaxCandidates * 5);
  if (attr != hipSuccess) return attr;
  const unsigned groups = unsigned((a.NT + a.G - 1) / a.G);
  const unsigned blocks = unsigned(a.B) * unsigned(a.H) * groups;
  topk_lists_kernel<<<blocks, kThreads, lds_bytes, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
