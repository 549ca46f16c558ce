// kv_append: copy the current chunk's K and V into the pages of one window slot.
//
// Appending the new chunk's keys and values to the layer's KV cache is the
// cache side of chunk-wise streaming generation (Sec. 2.3.2, dynamic cache
// management; Alg. 3, inference part).  One workgroup fills one page
// (slot, b, h, tile t): K is copied row for row (16-byte loads and stores); V
// is staged in LDS and written transposed with the keys of every group of 16
// stored in swap23 order, which is the order in which the attention kernel's
// 32x32x16 MFMA consumes them.  128-token pages store both as blocks of 64
// columns (K: [2][T][64], dimension halves; V^T: [2][D][64], key halves), so
// that 64 keys of either are 8 KB pieces of 128-byte rows; 64-token pages keep
// K as [T][D] and V^T as [D][T].  Rows past the chunk end get
// the pad value.  The page's pooled key (the block-mean pooling of Eq. 4,
// Sec. 2.3.1 (b)) is written beside it: the float32 mean of the valid K rows,
// summed in token order and divided once by their count, so that the top-k
// list builder ranks tiles with a fixed arithmetic.  HBM-bound: 2*B*L*H*D*2
// bytes read, 2*B*NT*T*H*D*2 + B*NT*H*D*4 written.
#include "../launch.h"

namespace uf {
namespace {

constexpr int kD = 128;
constexpr int kThreads = 256;

template <int T>
__global__ __launch_bounds__(kThreads) void kv_append_kernel(AppendArgs a) {
  constexpr int kRowChunks = kD / 8;          // 16-byte chunks per K/V input row
  constexpr int kStage = kRowChunks + 1;      // LDS row stride in chunks (272 bytes)
  constexpr bool kBlocks = T == 128;          // 64-column blocks (see above)
  __shared__ uint4 vstage[T * kStage];

  const int page = blockIdx.x;                // (b*H + h)*NT + t
  const int t = page % a.NT;
  const int bh = page / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int valid = tile_valid(a.tv, t, a.NT, a.tail, T);

  uint8_t* dst = a.pool + (size_t(a.slot) * a.B * a.H * a.NT + size_t(page)) * page_bytes(T, kD);
  uint4 pad;
  pad.x = pad.y = pad.z = pad.w = uint32_t(a.pad) | (uint32_t(a.pad) << 16);

  uint4* kdst = reinterpret_cast<uint4*>(dst);
  for (int c = threadIdx.x; c < T * kRowChunks; c += kThreads) {
    const int r = c / kRowChunks;
    const int cc = c % kRowChunks;
    uint4 kk = pad, vv = pad;
    if (r < valid) {
      const size_t off = ((size_t(b) * a.L + size_t(t) * T + r) * a.H + h) * kD + cc * 8;
      kk = *reinterpret_cast<const uint4*>(a.k + off);
      vv = *reinterpret_cast<const uint4*>(a.v + off);
    }
    kdst[kBlocks ? (cc >> 3) * (T * 8) + r * 8 + (cc & 7) : c] = kk;
    vstage[r * kStage + cc] = vv;
  }
  __syncthreads();

  const uint16_t* vs = reinterpret_cast<const uint16_t*>(vstage);
  uint4* vdst = reinterpret_cast<uint4*>(dst + size_t(T) * kD * 2);
  constexpr int kOutChunks = T / 8;           // 16-byte chunks per V^T row
  for (int c = threadIdx.x; c < kD * kOutChunks; c += kThreads) {
    const int d = c / kOutChunks;
    const int p0 = (c % kOutChunks) * 8;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = vs[swap23(p0 + 2 * e) * (kStage * 8) + d];
      const uint32_t hi = vs[swap23(p0 + 2 * e + 1) * (kStage * 8) + d];
      w[e] = lo | (hi << 16);
    }
    vdst[kBlocks ? (p0 >> 6) * (kD * 8) + d * 8 + ((p0 & 63) >> 3) : c] = make_uint4(w[0], w[1], w[2], w[3]);
  }

  // Pooled key: the valid K rows are staged again (L2-resident since the
  // copy above read them) in the V stage, then lane d adds column d in order.
  __syncthreads();
  for (int c = threadIdx.x; c < valid * kRowChunks; c += kThreads) {
    const int r = c / kRowChunks;
    const int cc = c % kRowChunks;
    const size_t off = ((size_t(b) * a.L + size_t(t) * T + r) * a.H + h) * kD + cc * 8;
    vstage[r * kStage + cc] = *reinterpret_cast<const uint4*>(a.k + off);
  }
  __syncthreads();
  if (threadIdx.x < kD) {
    const int d = threadIdx.x;
    float acc = 0.f;
#pragma unroll 8
    for (int r = 0; r < valid; ++r) acc += __uint_as_float(uint32_t(vs[r * (kStage * 8) + d]) << 16);
    a.kmean[(size_t(a.slot) * a.B * a.H * a.NT + size_t(page)) * kD + d] = acc / float(valid);
  }
}

}  // namespace

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream) {
  const unsigned blocks = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  if (a.T == 128)
    kv_append_kernel<128><<<blocks, kThreads, 0, stream>>>(a);
  else
    kv_append_kernel<64><<<blocks, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
