// attn_fwd: block-sparse chunk-causal attention forward on gfx950.
//
// For one (b, h, query tile i) the workgroup walks the kept key tiles of its
// list in ascending logical order (Eq. 4: attention restricted to the kept
// blocks of the chunk-causal window) and keeps an online softmax.
//
// Work split: 32 queries per wave, T/32 waves per workgroup.  The kernel
// computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (K from LDS as the A
// operand, Q held in registers as the B operand), so in the result layout
// every lane owns one query column and 16 key rows per 32-key block; the row
// max and row sum need one exchange with the partner lane (permlane32 swap).
// The exponentiated scores are rounded to bf16 in place and reused directly as
// the B operand of O^T += V^T P^T; V pages are stored transposed with the keys
// of each group of 16 in swap23 order, which is exactly the k-slot order in
// which the S^T result lanes hold them.  Softmax runs in base 2 with
// scale*log2(e) folded into one FMA.  fp32 accumulation throughout; O is
// normalised once at the end and rounded to bf16 (nearest even).
#include "../launch.h"

namespace uf {
namespace {

constexpr int kD = 128;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Both lanes of a pair (l, l^32) get the same value.
__device__ inline float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return uint32_t(__builtin_bit_cast(uint16_t, a)) | (uint32_t(__builtin_bit_cast(uint16_t, b)) << 16);
}

template <int T>
__global__ __launch_bounds__(T * 2) void attn_fwd_kernel(AttnArgs a) {
  constexpr int kWaves = T / 32;
  constexpr int kThreads = kWaves * 64;
  constexpr int KB = T / 32;              // 32-key blocks per key tile
  constexpr int kKChunks = kD / 8;        // 16-byte chunks per K row
  constexpr int kVChunks = T / 8;         // 16-byte chunks per V^T row
  __shared__ uint4 sK[T * kKChunks];
  __shared__ uint4 sV[kD * kVChunks];

  const int row = blockIdx.x;
  const int qt = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int g = lane >> 5;
  const int ln = lane & 31;
  const int qrow = qt * T + wave * 32 + ln;
  const bool qvalid = qrow < a.L;

  // Q^T as the B operand: lane holds query ln, dims 16*ks + 8*g .. +8.
  bf16x8 qf[kD / 16];
  {
    const uint16_t* qp = a.q + ((size_t(b) * a.L + (qvalid ? qrow : 0)) * a.H + h) * kD + 8 * g;
#pragma unroll
    for (int ks = 0; ks < kD / 16; ++ks) {
      uint4 u = make_uint4(0, 0, 0, 0);
      if (qvalid) u = *reinterpret_cast<const uint4*>(qp + 16 * ks);
      qf[ks] = as_bf16x8(u);
    }
  }

  f32x16 o[kD / 32];
#pragma unroll
  for (int mb = 0; mb < kD / 32; ++mb) o[mb] = f32x16{};
  float m = -INFINITY;   // running max of raw scores q.k
  float l = 0.f;         // running sum of exp(scale * (s - m))

  const int count = a.counts[row];
  const int32_t* list = a.idx + size_t(row) * a.nk_cap;
  const size_t pbytes = page_bytes(T, kD);
  const float c2 = a.scale_log2;

  for (int n = 0; n < count; ++n) {
    const int j = list[n];
    if (unsigned(j) >= unsigned(a.nk)) continue;   // stale entry: outside the window
    const int pos = j / a.NT;
    const int t = j - pos * a.NT;
    const uint4* page = reinterpret_cast<const uint4*>(
        a.pool + ((size_t(a.slot_of[pos]) * a.B + b) * a.H + h) * a.NT * pbytes + size_t(t) * pbytes);
    const int valid = (t == a.NT - 1) ? a.tail : T;

    __syncthreads();
    for (int c = tid; c < T * kKChunks; c += kThreads) {
      const int r = c / kKChunks, cc = c % kKChunks;
      sK[r * kKChunks + (cc ^ (r & 15))] = page[c];
    }
    for (int c = tid; c < kD * kVChunks; c += kThreads) {
      const int d = c / kVChunks, cc = c % kVChunks;
      sV[d * kVChunks + (cc ^ (d & (kVChunks - 1)))] = page[T * kKChunks + c];
    }
    __syncthreads();

    // S^T = K Q^T : KB blocks of 32 keys x 32 queries.
    f32x16 s[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      s[kb] = f32x16{};
      const int r = kb * 32 + ln;
#pragma unroll
      for (int ks = 0; ks < kD / 16; ++ks) {
        const int cc = 2 * ks + g;
        const bf16x8 kf = as_bf16x8(sK[r * kKChunks + (cc ^ (r & 15))]);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[kb], 0, 0, 0);
      }
    }

    // Padding keys of a chunk's last tile never count.
    if (valid < T) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = kb * 32 + 8 * (e >> 2) + 4 * g + (e & 3);
          if (key >= valid) s[kb][e] = -INFINITY;
        }
    }

    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kb][e]);
    mx = pair_max(mx);
    const float mnew = fmaxf(m, mx);
    const float alpha = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((m - mnew) * c2);
    const float mb2 = mnew * c2;
    float rs = 0.f;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][e], c2, -mb2));
        s[kb][e] = p;
        rs += p;
      }
    rs = pair_sum(rs);
    l = l * alpha + rs;
    m = mnew;
#pragma unroll
    for (int mb = 0; mb < kD / 32; ++mb) o[mb] *= alpha;

    // P^T as the B operand: 16-key halves of each 32-key block.
    bf16x8 pf[KB][2];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        uint4 u;
        u.x = pack_bf16x2(s[kb][8 * hh + 0], s[kb][8 * hh + 1]);
        u.y = pack_bf16x2(s[kb][8 * hh + 2], s[kb][8 * hh + 3]);
        u.z = pack_bf16x2(s[kb][8 * hh + 4], s[kb][8 * hh + 5]);
        u.w = pack_bf16x2(s[kb][8 * hh + 6], s[kb][8 * hh + 7]);
        pf[kb][hh] = as_bf16x8(u);
      }

    // O^T += V^T P^T : 4 blocks of 32 dims x 32 queries.
#pragma unroll
    for (int mb = 0; mb < kD / 32; ++mb) {
      const int d = mb * 32 + ln;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int cc = 2 * (2 * kb + hh) + g;
          const bf16x8 vf = as_bf16x8(sV[d * kVChunks + (cc ^ (d & (kVChunks - 1)))]);
          o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kb][hh], o[mb], 0, 0, 0);
        }
    }
  }

  if (qvalid) {
    const float inv = (l > 0.f) ? 1.f / l : 0.f;
    uint16_t* op = a.o + ((size_t(b) * a.L + qrow) * a.H + h) * kD;
#pragma unroll
    for (int mb = 0; mb < kD / 32; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = mb * 32 + 8 * i + 4 * g;
        uint2 u;
        u.x = pack_bf16x2(o[mb][4 * i + 0] * inv, o[mb][4 * i + 1] * inv);
        u.y = pack_bf16x2(o[mb][4 * i + 2] * inv, o[mb][4 * i + 3] * inv);
        *reinterpret_cast<uint2*>(op + d0) = u;
      }
    if (a.lse != nullptr && g == 0)
      a.lse[(size_t(b) * a.H + h) * a.L + qrow] = (l > 0.f) ? m * a.scale + logf(l) : -INFINITY;
  }
}

}  // namespace

hipError_t launch_attn_fwd(const AttnArgs& a, hipStream_t stream) {
  const unsigned blocks = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  if (a.T == 128)
    attn_fwd_kernel<128><<<blocks, 256, 0, stream>>>(a);
  else
    attn_fwd_kernel<64><<<blocks, 128, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
