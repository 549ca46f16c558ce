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
// Two kernels.  pool_queries: one workgroup per query tile stages the tile's
// valid rows in LDS and lane d adds column d in token order, writing the
// pooled query into the list buffer's scratch section.  topk_lists: one
// workgroup of 256 lanes per (b, h, group of G query tiles); a lane takes one
// ranked candidate at a time, loads its pooled key (512 bytes, L2-resident)
// into registers and scores it against the G pooled queries held in LDS.  The
// selection of a row runs in one wave: a radix select over the order keys
// (four passes of 8-bit histograms in LDS) finds the budget-th largest key,
// then one ballot pass over the candidates in index order keeps every larger
// key and the first equal keys the budget still admits (ties to the lower
// index).  Each row is then written by the shared output stage.
#include "list_emit.h"

#pragma clang fp contract(off)

namespace uf {
namespace {

using lists::kThreads;
using lists::kWaves;
constexpr int kD = 128;
constexpr int kMaxG = 8;

__device__ inline float bf16_to_f32(uint16_t x) { return __uint_as_float(uint32_t(x) << 16); }

// Unsigned key that orders float32 values like the real line.
__device__ inline uint32_t order_key(float s) {
  const uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int T>
__global__ __launch_bounds__(kThreads) void pool_queries_kernel(TopkArgs a) {
  __shared__ uint4 stage[T * (kD / 8)];
  const int row = blockIdx.x;            // (b*H + h)*NT + i
  const int i = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int nv = tile_valid(a.tv, i, a.NT, a.tail, T);
  for (int c = threadIdx.x; c < nv * (kD / 8); c += kThreads) {
    const int r = c / (kD / 8);
    const int cc = c - r * (kD / 8);
    stage[c] = *reinterpret_cast<const uint4*>(a.q + ((size_t(b) * a.L + size_t(i) * T + r) * a.H + h) * kD + cc * 8);
  }
  __syncthreads();
  if (threadIdx.x < kD) {
    const uint16_t* st = reinterpret_cast<const uint16_t*>(stage);
    const int d = threadIdx.x;
    float acc = 0.f;
#pragma unroll 8
    for (int r = 0; r < nv; ++r) acc += bf16_to_f32(st[r * kD + d]);
    float* qmean = reinterpret_cast<float*>(a.lists + a.scratch_offset);
    qmean[size_t(row) * kD + d] = acc / float(nv);
  }
}

__global__ __launch_bounds__(kThreads) void topk_lists_kernel(TopkArgs a) {
  extern __shared__ uint32_t dyn[];
  __shared__ float qm[kMaxG][kD];
  __shared__ uint32_t whist[kWaves][256];
  __shared__ int wave_count[kWaves];

  const int nc = max(a.cand_hi - a.cand_lo, 0);   // ranked candidates of a row
  uint32_t* keys = dyn;                            // [G][nc]
  uint8_t* sel = reinterpret_cast<uint8_t*>(dyn + size_t(a.G) * nc);   // [G][nc]

  const int groups = (a.NT + a.G - 1) / a.G;
  const int grp = blockIdx.x % groups;
  const int bh = blockIdx.x / groups;
  const int i0 = grp * a.G;
  const int gn = min(a.G, a.NT - i0);
  const int tid = threadIdx.x;

  // 1. pooled queries of the group
  const float* qmean = reinterpret_cast<const float*>(a.lists + a.scratch_offset);
  for (int e = tid; e < gn * kD; e += kThreads) qm[e / kD][e % kD] = qmean[(size_t(bh) * a.NT + i0) * kD + e];
  __syncthreads();

  // 2. scores: lane takes candidate m, its pooled key in registers
  const size_t slot_pages = size_t(a.B) * a.H * a.NT;
  const size_t head_page = size_t(bh) * a.NT;
  for (int m = tid; m < nc; m += kThreads) {
    const int j = a.cand_lo + m;
    const int pos = j / a.NT;
    const int t = j - pos * a.NT;
    const float4* kp = reinterpret_cast<const float4*>(a.kmean + (size_t(a.slot_of[pos]) * slot_pages + head_page + t) * kD);
    float4 k4[kD / 4];
#pragma unroll
    for (int c = 0; c < kD / 4; ++c) k4[c] = kp[c];
    for (int g = 0; g < gn; ++g) {
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < kD / 4; ++c) {
        acc = acc + qm[g][4 * c + 0] * k4[c].x;
        acc = acc + qm[g][4 * c + 1] * k4[c].y;
        acc = acc + qm[g][4 * c + 2] * k4[c].z;
        acc = acc + qm[g][4 * c + 3] * k4[c].w;
      }
      keys[size_t(g) * nc + m] = order_key(acc);
    }
  }
  __syncthreads();

  // 3. selection, one wave per row
  {
    const int wave = tid >> 6;
    const int lane = tid & 63;
    uint32_t* hist = whist[wave];
    for (int g = wave; g < gn; g += kWaves) {
      const uint32_t* row = keys + size_t(g) * nc;
      uint8_t* sg = sel + size_t(g) * nc;
      if (a.budget >= nc || a.budget == 0) {
        for (int m = lane; m < nc; m += 64) sg[m] = a.budget > 0 ? 1 : 0;
        continue;
      }
      // radix select: `need` = rank of the wanted key among keys matching `prefix` on `pmask`
      uint32_t prefix = 0, pmask = 0;
      int need = a.budget;
      for (int shift = 24; shift >= 0; shift -= 8) {
        for (int e = lane; e < 256; e += 64) hist[e] = 0;
        __builtin_amdgcn_wave_barrier();
        for (int m = lane; m < nc; m += 64) {
          const uint32_t k = row[m];
          if ((k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
        }
        __builtin_amdgcn_wave_barrier();
        // lane l holds bins 255-4l .. 252-4l (descending); exclusive prefix over lanes
        uint32_t hb[4];
        uint32_t own = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          hb[e] = hist[255 - 4 * lane - e];
          own += hb[e];
        }
        uint32_t incl = own;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t y = __shfl_up(incl, o);
          if (lane >= o) incl += y;
        }
        const uint32_t excl = incl - own;
        // the lane whose bins cover rank `need`
        const bool mine = excl < uint32_t(need) && uint32_t(need) <= incl;
        const int owner = __ffsll(static_cast<long long>(__ballot(mine))) - 1;
        int bin = 0;
        uint32_t above = excl;
        if (mine) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (above + hb[e] >= uint32_t(need)) {
              bin = 255 - 4 * lane - e;
              break;
            }
            above += hb[e];
          }
        }
        bin = __shfl(bin, owner);
        above = __shfl(above, owner);
        prefix |= uint32_t(bin) << shift;
        pmask |= 255u << shift;
        need -= int(above);
        __builtin_amdgcn_wave_barrier();
      }
      // keys above the threshold, and the first `need` keys equal to it in index order
      int taken = 0;
      for (int m0 = 0; m0 < nc; m0 += 64) {
        const int m = m0 + lane;
        const uint32_t k = (m < nc) ? row[m] : 0u;
        const bool eq = (m < nc) && k == prefix;
        const uint64_t eqb = __ballot(eq);
        const int rank = taken + __popcll(eqb & ((1ull << lane) - 1ull));
        if (m < nc) sg[m] = (k > prefix || (eq && rank < need)) ? 1 : 0;
        taken += __popcll(eqb);
      }
    }
  }
  __syncthreads();

  // 4. the list rows
  int32_t* counts = reinterpret_cast<int32_t*>(a.lists);
  for (int g = 0; g < gn; ++g) {
    const int row = bh * a.NT + i0 + g;
    int32_t* idx = reinterpret_cast<int32_t*>(a.lists + a.idx_offset) + size_t(row) * a.nk_cap;
    uint32_t* mask = reinterpret_cast<uint32_t*>(a.lists + a.mask_offset) + size_t(row) * a.mask_words;
    const uint8_t* sg = sel + size_t(g) * nc;
    const int qi = i0 + g;
    auto keep_of = [&](int j) {
      if (j >= a.nk) return false;
      if (!tile_local(a.tv, qi, j % a.NT)) return false;   // structural local window (block geometry)
      if (j < a.cand_lo || j >= a.cand_hi) return true;    // forced: pinned or current chunk
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
  const unsigned rows = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  if (a.T == 128)
    pool_queries_kernel<128><<<rows, kThreads, 0, stream>>>(a);
  else
    pool_queries_kernel<64><<<rows, kThreads, 0, stream>>>(a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned groups = unsigned((a.NT + a.G - 1) / a.G);
  const unsigned blocks = unsigned(a.B) * unsigned(a.H) * groups;
  topk_lists_kernel<<<blocks, kThreads, lds_bytes, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
