// block_permute: reorder token rows between raster order and 3-D block order.
//
// The (t, h, w) token grid of a chunk is divided into (bt, bh, bw) blocks
// (Sec. 2.3.1 (a)); in block order every block owns one tile of bt*bh*bw rows
// holding its valid tokens in raster (t, h, w) order, then padding rows.  One
// workgroup per (b, block, head) copies the block's rows of that head, 128
// bf16 each (16-byte chunks): forward writes zero padding rows, inverse drops
// them.  HBM-bound.
#include "../launch.h"

namespace uf {
namespace {

constexpr int kThreads = 256;
constexpr int kRowChunks = 16;   // 16-byte chunks per (token, head) row of 128 bf16

__global__ __launch_bounds__(kThreads) void block_permute_kernel(PermuteArgs a) {
  const int nb = (a.frames + a.bt - 1) / a.bt * a.nbh * a.nbw;
  const int head = blockIdx.x % a.H;
  const int blk = (blockIdx.x / a.H) % nb;
  const int b = blockIdx.x / a.H / nb;
  const int bti = blk / (a.nbh * a.nbw);
  const int bhi = (blk / a.nbw) % a.nbh;
  const int bwi = blk % a.nbw;
  const int nt = min(a.bt, a.frames - bti * a.bt);
  const int nh = min(a.bh, a.gh - bhi * a.bh);
  const int nw = min(a.bw, a.gw - bwi * a.bw);
  const int valid = nt * nh * nw;
  const int tile = a.bt * a.bh * a.bw;
  const int per_row = a.H * kRowChunks;
  const uint4* src = reinterpret_cast<const uint4*>(a.src);
  uint4* dst = reinterpret_cast<uint4*>(a.dst);
  for (int c = threadIdx.x; c < tile * kRowChunks; c += kThreads) {
    const int r = c / kRowChunks;
    const int cc = head * kRowChunks + (c - r * kRowChunks);
    const size_t brow = size_t(b) * a.padded + size_t(blk) * tile + r;   // block-order row
    if (r < valid) {
      const int dt = r / (nh * nw);
      const int dh = (r / nw) % nh;
      const int dw = r % nw;
      const size_t tok = (size_t(bti * a.bt + dt) * a.gh + bhi * a.bh + dh) * a.gw + bwi * a.bw + dw;
      const size_t rrow = size_t(b) * a.tokens + tok;                      // raster row
      if (a.inverse)
        dst[rrow * per_row + cc] = src[brow * per_row + cc];
      else
        dst[brow * per_row + cc] = src[rrow * per_row + cc];
    } else if (!a.inverse) {
      dst[brow * per_row + cc] = make_uint4(0, 0, 0, 0);
    }
  }
}

}  // namespace

hipError_t launch_block_permute(const PermuteArgs& a, hipStream_t stream) {
  const unsigned nb = unsigned((a.frames + a.bt - 1) / a.bt * a.nbh * a.nbw);
  block_permute_kernel<<<unsigned(a.B) * nb * unsigned(a.H), kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
