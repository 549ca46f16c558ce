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
// Sec. 2.3.1 (b)) is written beside it: the float32 mean of the valid K rows
// (staged in LDS from the registers of the copy, so K is read once), summed
// in token order and divided once by their count, so that the top-k list
// builder ranks tiles with a fixed arithmetic.  HBM-bound: 2*B*L*H*D*2
// bytes read, 2*B*NT*T*H*D*2 + B*NT*H*D*4 written.
#include "../launch.h"

namespace uf {
namespace {

constexpr int kD = 128;
constexpr int kThreads = 256;

template <int T>
__global__ __launch_bounds__(kThreads) void kv_append_kernel(AppendArgs a) {
  constexpr int kRowChunks = kD / 8;          // 16-byte chunks per K/V input row
  constexpr int kStage = kRowChunks + 1;      // V stage row stride in chunks (272 bytes)
  constexpr int kPer = T * kRowChunks / kThreads;   // chunks of K (and of V) per thread
  constexpr int kRowStep = kThreads / kRowChunks;   // rows between a thread's chunks
  constexpr bool kBlocks = T == 128;          // 64-column blocks (see above)
  // V rows at a 272-byte stride for the transposed writes, then, reused, K
  // rows at 256 bytes for the pooled key (35 KB: four workgroups per CU)
  __shared__ uint4 stage[T * kStage];

  const int page = blockIdx.x;                // (b*H + h)*NT + t
  const int t = page % a.NT;
  const int bh = page / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int valid = tile_valid(a.tv, t, a.NT, a.tail, T);

  uint8_t* dst = a.pool + (size_t(a.slot) * a.B * a.H * a.NT + size_t(page)) * page_bytes(T, kD);
  uint4 pad;
  pad.x = pad.y = pad.z = pad.w = uint32_t(a.pad) | (uint32_t(a.pad) << 16);

  // Every load of the thread is issued before any store: the stores could
  // alias the inputs as far as the compiler knows, so loads interleaved with
  // them would each wait for a full memory round trip.
  const int cc = threadIdx.x % kRowChunks;    // the thread's 16-byte column chunk
  const int r0 = threadIdx.x / kRowChunks;    // its rows: r0 + kRowStep * i
  uint4 kk[kPer], vv[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int r = r0 + kRowStep * i;
    kk[i] = pad;
    vv[i] = pad;
    if (r < valid) {
      const size_t off = ((size_t(b) * a.L + size_t(t) * T + r) * a.H + h) * kD + cc * 8;
      kk[i] = *reinterpret_cast<const uint4*>(a.k + off);
      vv[i] = *reinterpret_cast<const uint4*>(a.v + off);
    }
  }
  uint4* kdst = reinterpret_cast<uint4*>(dst);
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int r = r0 + kRowStep * i;
    kdst[kBlocks ? (cc >> 3) * (T * 8) + r * 8 + (cc & 7) : r * kRowChunks + cc] = kk[i];
    stage[r * kStage + cc] = vv[i];
  }
  __syncthreads();

  const uint16_t* vs = reinterpret_cast<const uint16_t*>(stage);
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

  // Pooled key: the K rows (still in registers) are staged in the same LDS,
  // then lane d adds column d in token order.
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kPer; ++i) stage[(r0 + kRowStep * i) * kRowChunks + cc] = kk[i];
  __syncthreads();
  if (threadIdx.x < kD) {
    const int d = threadIdx.x;
    const uint16_t* ks = reinterpret_cast<const uint16_t*>(stage);
    float acc = 0.f;
#pragma unroll 8
    for (int r = 0; r < valid; ++r) acc += __uint_as_float(uint32_t(ks[r * kD + d]) << 16);
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
