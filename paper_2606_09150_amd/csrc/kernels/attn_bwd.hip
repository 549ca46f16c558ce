// attn_bwd: gradients of the block-sparse chunk-causal attention.
//
// The student of Phase I is trained through the sparse causal attention of
// Sec. 2.3.1 (the Eq. 4 mask inside the generator that the DMD objective
// updates), so the training side needs dQ, dK and dV over the same keep
// lists.  With p = exp(scale*q.k - lse) over the kept keys of a row,
// delta = <dO, O>, dS = P (dO V^T - delta):
//   dV = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K.
//
// Four kernels, all with 32x32x16 bf16 MFMA and fp32 accumulation:
//  * prep_queries: per query tile, Q and dO row-major and transposed (query
//    index in swap23 order within groups of 16, the k-slot order of the MFMA
//    result lanes), LSE*log2(e) (+inf for rows past the chunk end, so that their
//    weights vanish) and delta;
//  * prep_keys: per window key tile, K^T (keys in swap23 order) and V
//    row-major, from the pool's K rows and V^T columns;
//  * dkdv: one workgroup per window key tile, four waves of 32 keys; it walks
//    the query tiles whose lists keep the tile (mask bits), and per 32-query
//    block computes S = Q K^T (keys on the result lanes), P, dP = dO V^T,
//    dS, then dV^T += dO^T P and dK^T += Q^T dS with P and dS used in place as
//    B operands;
//  * dq: one workgroup per query tile, four waves of 32 queries; it walks the
//    row's list and per 32-key block computes S^T = K Q^T (queries on the
//    lanes), P^T, dP^T = V dO^T, dS^T, then dQ^T += K^T dS^T.
// No atomics: every output row is owned by one workgroup, so results are
// reproducible.  Tiles stream into LDS by direct global->LDS copies with the
// same XOR swizzle as the forward; the loops are single-buffered.
#include "attn_common.h"

namespace uf {
namespace {

using namespace attn;

constexpr int kT = 128;
constexpr int kThreads = 256;                  // four waves
constexpr uint32_t kTile = 32768;              // one [128][128] bf16 tile
constexpr int kStage = 17;                     // padded LDS row stride in 16-byte chunks

__device__ inline float bf16f(uint16_t x) { return __uint_as_float(uint32_t(x) << 16); }
__device__ inline uint16_t f2bf(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

// ---------------------------------------------------------------- prep ----

// Row-major copy of one query tile of x [B, L, H, D] into dst (rows past the
// chunk end zero) and into an LDS stage; then the transposed tile.
__device__ void tile_both_ways(const uint16_t* x, int b, int h, int i, int nv, const BwdArgs& a, uint4* stage,
                               uint4* dst_rows, uint4* dst_t) {
  for (int c = threadIdx.x; c < kT * 16; c += kThreads) {
    const int r = c >> 4, cc = c & 15;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r < nv) v = *reinterpret_cast<const uint4*>(x + ((size_t(b) * a.L + size_t(i) * kT + r) * a.H + h) * kD + cc * 8);
    dst_rows[c] = v;
    stage[r * kStage + cc] = v;
  }
  __syncthreads();
  const uint16_t* st = reinterpret_cast<const uint16_t*>(stage);
  for (int c = threadIdx.x; c < kD * 16; c += kThreads) {
    const int d = c >> 4, p0 = (c & 15) * 8;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = st[swap23(p0 + 2 * e) * (kStage * 8) + d];
      const uint32_t hi = st[swap23(p0 + 2 * e + 1) * (kStage * 8) + d];
      w[e] = lo | (hi << 16);
    }
    dst_t[c] = make_uint4(w[0], w[1], w[2], w[3]);
  }
  __syncthreads();
}

__global__ __launch_bounds__(kThreads) void bwd_prep_queries_kernel(BwdArgs a) {
  __shared__ uint4 stage[kT * kStage];
  const int row = blockIdx.x;                  // (b*H + h)*NT + i
  const int i = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H, b = bh / a.H;
  const int nv = tile_valid(a.tv, i, a.NT, a.tail, kT);
  uint8_t* qt = a.work + size_t(row) * kBwdQTile;
  tile_both_ways(a.q, b, h, i, nv, a, stage, reinterpret_cast<uint4*>(qt), reinterpret_cast<uint4*>(qt + kTile));
  tile_both_ways(a.dout, b, h, i, nv, a, stage, reinterpret_cast<uint4*>(qt + 2 * kTile),
                 reinterpret_cast<uint4*>(qt + 3 * kTile));
  float* lse2 = reinterpret_cast<float*>(qt + 4 * kTile);
  float* delta = lse2 + kT;
  if (threadIdx.x < kT) {
    const int q = threadIdx.x;
    float l2 = INFINITY, dl = 0.f;
    if (q < nv) {
      const size_t tok = size_t(i) * kT + q;
      l2 = a.lse[(size_t(b) * a.H + h) * a.L + tok] * 1.4426950408889634f;
      const uint16_t* op = a.o + ((size_t(b) * a.L + tok) * a.H + h) * kD;
      const uint16_t* gp = a.dout + ((size_t(b) * a.L + tok) * a.H + h) * kD;
      for (int d = 0; d < kD; ++d) dl += bf16f(op[d]) * bf16f(gp[d]);
    }
    lse2[q] = l2;
    delta[q] = dl;
  }
}

__global__ __launch_bounds__(kThreads) void bwd_prep_keys_kernel(BwdArgs a) {
  __shared__ uint4 stage[kT * kStage];
  const int kj = blockIdx.x;                   // ((pos*B + b)*H + h)*NT + t
  const int t = kj % a.NT;
  const int posbh = kj / a.NT;
  const int bh = posbh % (a.B * a.H);
  const int pos = posbh / (a.B * a.H);
  const uint8_t* page = a.pool + ((size_t(a.slot_of[pos]) * a.B * a.H + bh) * a.NT + t) * page_bytes(kT, kD);
  uint8_t* kt = a.work + size_t(a.B) * a.H * a.NT * kBwdQTile + size_t(kj) * kBwdKTile;
  const uint4* krows = reinterpret_cast<const uint4*>(page);
  const uint4* vt = reinterpret_cast<const uint4*>(page + kTile);
  // K^T: stage the K rows, write columns with keys in swap23 order
  for (int c = threadIdx.x; c < kT * 16; c += kThreads) stage[(c >> 4) * kStage + (c & 15)] = krows[c];
  __syncthreads();
  const uint16_t* st = reinterpret_cast<const uint16_t*>(stage);
  uint4* dst = reinterpret_cast<uint4*>(kt);
  for (int c = threadIdx.x; c < kD * 16; c += kThreads) {
    const int d = c >> 4, p0 = (c & 15) * 8;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = st[swap23(p0 + 2 * e) * (kStage * 8) + d];
      const uint32_t hi = st[swap23(p0 + 2 * e + 1) * (kStage * 8) + d];
      w[e] = lo | (hi << 16);
    }
    dst[c] = make_uint4(w[0], w[1], w[2], w[3]);
  }
  __syncthreads();
  // V rows: V^T row d holds key swap23(p) at column p
  for (int c = threadIdx.x; c < kD * 16; c += kThreads) stage[(c >> 4) * kStage + (c & 15)] = vt[c];
  __syncthreads();
  dst = reinterpret_cast<uint4*>(kt + kTile);
  for (int c = threadIdx.x; c < kT * 16; c += kThreads) {
    const int key = c >> 4, d0 = (c & 15) * 8;
    const int p = swap23(key);
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = st[(d0 + 2 * e) * (kStage * 8) + p];
      const uint32_t hi = st[(d0 + 2 * e + 1) * (kStage * 8) + p];
      w[e] = lo | (hi << 16);
    }
    dst[c] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// ------------------------------------------------------------- shared ----

// Copy one 32 KB tile global -> LDS with the forward's XOR swizzle (chunk c of
// row r lands at r*16 + (c ^ (r & 15))): eight 16-byte copies per wave.
__device__ inline void copy_tile(const uint8_t* src, uint32_t lds_tile, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int p = (4 * i + wave) * 64 + lane;
    const int r = p >> 4, cs = p & 15;
    dma16(src, uint32_t(r * 256 + ((cs ^ (r & 15)) * 16)), lds_tile + uint32_t(wave) * 1024u + uint32_t(i) * 4096u);
  }
}

// LDS byte offset of logical 16-byte chunk c of row r of a swizzled tile.
__device__ inline uint32_t swz(int r, int c) { return uint32_t(r * 256 + ((c ^ (r & 15)) * 16)); }

__device__ inline bf16x8 lds8(const uint8_t* base, uint32_t off) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(base + off));
}

// bf16 B operand for k-step kk (16 rows of a 32-row MFMA result block) from
// the fp32 result registers: rows 16kk + 8j + 4hl + i, j in {0, 1}, i in 0..3.
__device__ inline bf16x8 rows_to_operand(const f32x16& x, int kk) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)x[8 * kk + e];
  return r;
}

// ---------------------------------------------------------------- dkdv ----

__global__ __launch_bounds__(kThreads, 1) void bwd_dkdv_kernel(BwdArgs a) {
  __shared__ uint4 sQ[kT * 16], sQT[kT * 16], sO[kT * 16], sOT[kT * 16];
  __shared__ float sL[kT], sDl[kT];

  const int kj = blockIdx.x;                   // ((pos*B + b)*H + h)*NT + t
  const int t = kj % a.NT;
  const int posbh = kj / a.NT;
  const int bh = posbh % (a.B * a.H);
  const int pos = posbh / (a.B * a.H);
  const int h = bh % a.H, b = bh / a.H;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, hl = lane >> 5, ln = lane & 31;
  const int kvalid = tile_valid(a.tv, t, a.NT, a.tail, kT);
  const int key = wave * 32 + ln;               // this lane's key (result column)
  const bool key_ok = key < kvalid;
  const int j = pos * a.NT + t;                 // logical key tile

  // the wave's 32 keys as B operands: K rows from the page, V rows from the workspace
  const uint8_t* page = a.pool + ((size_t(a.slot_of[pos]) * a.B * a.H + bh) * a.NT + t) * page_bytes(kT, kD);
  const uint8_t* kw = a.work + size_t(a.B) * a.H * a.NT * kBwdQTile + size_t(kj) * kBwdKTile;
  bf16x8 kf[8], vf[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    kf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(page + size_t(key) * 256 + (2 * ks + hl) * 16));
    vf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(kw + kTile + size_t(key) * 256 + (2 * ks + hl) * 16));
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));

  f32x16 dvt[4], dkt[4];                        // [4 dim blocks][32 dims x 32 keys]
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
    dvt[mb] = f32x16{};
    dkt[mb] = f32x16{};
  }
  const uint8_t* lq = reinterpret_cast<const uint8_t*>(sQ);
  const uint8_t* lqt = reinterpret_cast<const uint8_t*>(sQT);
  const uint8_t* lo = reinterpret_cast<const uint8_t*>(sO);
  const uint8_t* lot = reinterpret_cast<const uint8_t*>(sOT);
  const float c2 = a.scale_log2;

  for (int i = 0; i < a.NT; ++i) {
    const int row = bh * a.NT + i;
    const uint32_t word = __builtin_amdgcn_readfirstlane(a.mask[size_t(row) * a.mask_words + (j >> 5)]);
    if (((word >> (j & 31)) & 1u) == 0) continue;
    const uint8_t* qt = a.work + size_t(row) * kBwdQTile;
    __syncthreads();                            // previous tiles consumed
    copy_tile(qt, lds_addr(sQ), wave, lane);
    copy_tile(qt + kTile, lds_addr(sQT), wave, lane);
    copy_tile(qt + 2 * kTile, lds_addr(sO), wave, lane);
    copy_tile(qt + 3 * kTile, lds_addr(sOT), wave, lane);
    if (tid < kT) {
      sL[tid] = reinterpret_cast<const float*>(qt + 4 * kTile)[tid];
      sDl[tid] = reinterpret_cast<const float*>(qt + 4 * kTile)[kT + tid];
    }
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
#pragma unroll 1
    for (int qb = 0; qb < 4; ++qb) {
      // S = Q K^T and dP = dO V^T for 32 queries x the wave's 32 keys
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const uint32_t off = swz(qb * 32 + ln, 2 * ks + hl);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(lq, off), kf[ks], s, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(lo, off), vf[ks], dp, 0, 0, 0);
      }
      // P and dS; result row r holds query qb*32 + 8*(r/4) + 4*hl + r%4
      f32x16 p, ds;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int q = qb * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
        const float e = __builtin_amdgcn_exp2f(s[r] * c2 - sL[q]);
        p[r] = key_ok ? e : 0.f;
        ds[r] = p[r] * (dp[r] - sDl[q]);
      }
      // dV^T += dO^T P, dK^T += Q^T dS (k = the block's queries)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 pb = rows_to_operand(p, kk);
        const bf16x8 db = rows_to_operand(ds, kk);
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
          const uint32_t off = swz(mb * 32 + ln, 4 * qb + 2 * kk + hl);
          dvt[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(lot, off), pb, dvt[mb], 0, 0, 0);
          dkt[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(lqt, off), db, dkt[mb], 0, 0, 0);
        }
      }
    }
  }

  // store: lane holds key `key`, dims mb*32 + 8*(r/4) + 4*hl + r%4; padding
  // rows inside the chunk (block order) get the zeros they accumulated
  const size_t tok = size_t(t) * kT + key;
  if (tok < size_t(a.L)) {
    const size_t base = (((size_t(pos) * a.B + b) * a.L + tok) * a.H + h) * kD;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = mb * 32 + 8 * g + 4 * hl;
        *reinterpret_cast<float4*>(a.dv + base + d0) =
            make_float4(dvt[mb][4 * g], dvt[mb][4 * g + 1], dvt[mb][4 * g + 2], dvt[mb][4 * g + 3]);
        *reinterpret_cast<float4*>(a.dk + base + d0) =
            make_float4(dkt[mb][4 * g] * a.scale, dkt[mb][4 * g + 1] * a.scale, dkt[mb][4 * g + 2] * a.scale,
                        dkt[mb][4 * g + 3] * a.scale);
      }
  }
}

// ------------------------------------------------------------------ dq ----

__global__ __launch_bounds__(kThreads, 1) void bwd_dq_kernel(BwdArgs a) {
  __shared__ uint4 sK[kT * 16], sV[kT * 16], sKT[kT * 16];

  const int row = blockIdx.x;                  // (b*H + h)*NT + i
  const int i = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H, b = bh / a.H;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, hl = lane >> 5, ln = lane & 31;
  const int q = wave * 32 + ln;                 // this lane's query (result column)

  const uint8_t* qt = a.work + size_t(row) * kBwdQTile;
  bf16x8 qf[8], of[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    qf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qt + size_t(q) * 256 + (2 * ks + hl) * 16));
    of[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qt + 2 * kTile + size_t(q) * 256 + (2 * ks + hl) * 16));
  }
  const float l2 = reinterpret_cast<const float*>(qt + 4 * kTile)[q];
  const float dl = reinterpret_cast<const float*>(qt + 4 * kTile)[kT + q];
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));

  f32x16 dqt[4];                                // [4 dim blocks][32 dims x 32 queries]
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) dqt[mb] = f32x16{};
  const uint8_t* lk = reinterpret_cast<const uint8_t*>(sK);
  const uint8_t* lv = reinterpret_cast<const uint8_t*>(sV);
  const uint8_t* lkt = reinterpret_cast<const uint8_t*>(sKT);
  const float c2 = a.scale_log2;
  const int count = ((const const_i32*)a.counts)[row];
  const const_i32* list = ((const const_i32*)a.idx) + size_t(row) * a.nk_cap;
  const uint8_t* kbase = a.work + size_t(a.B) * a.H * a.NT * kBwdQTile;

  for (int n = 0; n < count; ++n) {
    const int j = list[n];
    if (unsigned(j) >= unsigned(a.nk)) continue;   // outside the window: no key
    const int pos = j / a.NT;
    const int t = j - pos * a.NT;
    const int kvalid = tile_valid(a.tv, t, a.NT, a.tail, kT);
    const uint8_t* page = a.pool + ((size_t(a.slot_of[pos]) * a.B * a.H + bh) * a.NT + t) * page_bytes(kT, kD);
    const uint8_t* kw = kbase + ((size_t(pos) * a.B * a.H + bh) * a.NT + t) * kBwdKTile;
    __syncthreads();                            // previous tiles consumed
    copy_tile(page, lds_addr(sK), wave, lane);
    copy_tile(kw + kTile, lds_addr(sV), wave, lane);
    copy_tile(kw, lds_addr(sKT), wave, lane);
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
#pragma unroll 1
    for (int kb = 0; kb < 4; ++kb) {
      // S^T = K Q^T and dP^T = V dO^T for the block's 32 keys x the wave's 32 queries
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const uint32_t off = swz(kb * 32 + ln, 2 * ks + hl);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(lk, off), qf[ks], s, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(lv, off), of[ks], dp, 0, 0, 0);
      }
      // result row r holds key kb*32 + 8*(r/4) + 4*hl + r%4
      f32x16 ds;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
        const float e = __builtin_amdgcn_exp2f(s[r] * c2 - l2);
        const float pr = key < kvalid ? e : 0.f;
        ds[r] = pr * (dp[r] - dl);
      }
      // dQ^T += K^T dS^T (k = the block's keys)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 db = rows_to_operand(ds, kk);
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
          dqt[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(lkt, swz(mb * 32 + ln, 4 * kb + 2 * kk + hl)), db,
                                                            dqt[mb], 0, 0, 0);
      }
    }
  }

  // padding rows inside the chunk accumulated zeros (their LSE is +inf)
  if (size_t(i) * kT + q < size_t(a.L)) {
    const size_t base = ((size_t(b) * a.L + size_t(i) * kT + q) * a.H + h) * kD;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = mb * 32 + 8 * g + 4 * hl;
        *reinterpret_cast<float4*>(a.dq + base + d0) =
            make_float4(dqt[mb][4 * g] * a.scale, dqt[mb][4 * g + 1] * a.scale, dqt[mb][4 * g + 2] * a.scale,
                        dqt[mb][4 * g + 3] * a.scale);
      }
  }
}

}  // namespace

hipError_t launch_attn_bwd(const BwdArgs& a, hipStream_t stream) {
  const unsigned qrows = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  const unsigned ktiles = unsigned(a.n_live) * qrows;
  bwd_prep_queries_kernel<<<qrows, kThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  bwd_prep_keys_kernel<<<ktiles, kThreads, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  bwd_dkdv_kernel<<<ktiles, kThreads, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  bwd_dq_kernel<<<qrows, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
