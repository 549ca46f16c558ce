// attn_bwd: gradients of the block-sparse chunk-causal attention.
//
// The student of Phase I is trained through the sparse causal attention of
// Sec. 2.3.1 (the Eq. 4 mask inside the generator that the DMD objective
// updates), so the training side needs dQ, dK and dV over the same keep
// lists.  With p = exp(scale*q.k - lse) over the kept keys of a row,
// delta = <dO, O>, dS = P (dO V^T - delta):
//   dV = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K.
//
// Three kernels, all with 32x32x16 bf16 MFMA and fp32 accumulation, each a
// template on the tile size T (128 or 64; the wave counts below are for 128
// and halve for 64):
//  * prep: per query tile, Q and dO rows (rows past the chunk end zero),
//    -LSE/scale (-inf on those rows, so that their weights vanish) and
//    -delta, which seed the S and dP accumulators;
//  * dkdv: one workgroup of eight waves per window key tile (one per CU).
//    Waves w and w + 4 share 32 keys.  The workgroup gathers the query tiles
//    whose mask bit keeps its tile and, per 32-query block, wave w computes
//    S = Q K^T and P, hands P to wave w + 4 through LDS and accumulates
//    dV^T += dO^T P, while wave w + 4 computes dP = dO V^T, dS = P (dP - delta)
//    from the shared P and accumulates dK^T += Q^T dS; the two run one block
//    apart, and the Q and dO rows of the next query tile are copied while the
//    current one is used;
//  * dq: one workgroup of four waves per query tile (two per CU), 32 queries
//    per wave; it walks the row's list and per 32-key block computes
//    S^T = K Q^T, dP^T = V dO^T, dS^T, then dQ^T += K^T dS^T.
// The transposed operands (dO^T, Q^T, K^T, and V rows from the pool's V^T)
// come from row-major LDS tiles through the transposing LDS read
// (ds_read_b64_tr_b16), so each tile is copied into LDS once, in the layout the
// pool or the workspace already holds.  No atomics: every output row is owned
// by one workgroup, so results are reproducible.
#include <mutex>
#include <type_traits>

#include "attn_common.h"
#include "../launch_bwd.h"

namespace uf {
namespace {

using namespace attn;

constexpr int kT = 128;
constexpr int kThreads = 256;                  // four waves
constexpr uint32_t kTile = 32768;              // one [128][128] bf16 tile

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) uint8_t lds_u8;

__device__ inline float bf16f(uint16_t x) { return __uint_as_float(uint32_t(x) << 16); }

// ---------------------------------------------------------------- prep ----

// T-token tiles; a record always has room for 128 rows and 128 per-query
// values, of which the first T are used.
template <int T>
__global__ __launch_bounds__(kThreads) void bwd_prep_kernel(BwdArgs a) {
  const int row = blockIdx.x;                  // (b*H + h)*NT + i
  const int i = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H, b = bh / a.H;
  const int nv = tile_valid(a.tv, i, a.NT, a.tail, T);
  uint8_t* rec = a.work + size_t(row) * kBwdQTile;
  uint4* qr = reinterpret_cast<uint4*>(rec);
  uint4* orow = reinterpret_cast<uint4*>(rec + kTile);
  for (int c = threadIdx.x; c < T * 16; c += kThreads) {
    const int r = c >> 4, cc = c & 15;
    uint4 vq = make_uint4(0, 0, 0, 0), vo = vq;
    if (r < nv) {
      const size_t off = ((size_t(b) * a.L + size_t(i) * T + r) * a.H + h) * kD + cc * 8;
      vq = *reinterpret_cast<const uint4*>(a.q + off);
      vo = *reinterpret_cast<const uint4*>(a.dout + off);
    }
    qr[c] = vq;
    orow[c] = vo;
  }
  float* nlse = reinterpret_cast<float*>(rec + 2 * kTile);
  float* ndelta = nlse + kT;
  if (threadIdx.x < T) {
    const int q = threadIdx.x;
    float nl = -INFINITY, dl = 0.f;
    if (q < nv) {
      const size_t tok = size_t(i) * T + q;
      nl = -a.lse[(size_t(b) * a.H + h) * a.L + tok] / a.scale;
      const uint16_t* op = a.o + ((size_t(b) * a.L + tok) * a.H + h) * kD;
      const uint16_t* gp = a.dout + ((size_t(b) * a.L + tok) * a.H + h) * kD;
      for (int d = 0; d < kD; ++d) dl += bf16f(op[d]) * bf16f(gp[d]);
    }
    nlse[q] = nl;
    ndelta[q] = -dl;
  }
}

// ------------------------------------------------------------- shared ----

// LDS layout of a [128][128] bf16 tile: 16-byte chunk c of row r sits at
// position perm(c) ^ f(r) of the row, perm swapping bits 1 and 3 of c and
// f(r) = (r3, r1, r0, r2 ^ r3) (bits 3..0).  Both 16-byte row reads (eight or
// sixteen consecutive rows, or rows in swap23 order, one chunk) and the
// transposing 8-byte reads (four consecutive rows, four consecutive chunks
// per 32 lanes) then touch every bank once per cycle, with 32 or 64 banks.
__device__ inline int swz_perm(int c) { return (c & ~10) | ((c & 2) << 2) | ((c & 8) >> 2); }
__device__ inline int swz_f(int r) { return (r & 8) | ((r & 3) << 1) | (((r >> 2) ^ (r >> 3)) & 1); }

// Copy one 32 KB K or V^T tile of a page global -> LDS in that layout: copy i
// of wave w fills LDS chunks [64*(4i + w), +64), i.e. row 16i + 4w + lane/16,
// position lane%16.  The row's low four bits do not depend on i, so one
// per-lane source offset serves all eight copies, with 2 KB steps on the
// scalar base: a page keeps the 16-byte chunks 0..7 and 8..15 of every row in
// two blocks of 128-byte rows, 16 KB apart.
__device__ inline uint32_t page_chunk(int r, int c) { return uint32_t((c >> 3) * 16384 + r * 128 + (c & 7) * 16); }
__device__ inline uint32_t copy_offset_page(int wave, int lane) {
  const int r = 4 * wave + (lane >> 4);
  return page_chunk(r, swz_perm((lane & 15) ^ swz_f(r)));
}
__device__ inline void copy_tile_page(const uint8_t* src, uint32_t lds_tile, uint32_t voff, int wave) {
#pragma unroll
  for (int i = 0; i < 8; ++i) dma16(src + i * 2048, voff, lds_tile + uint32_t(wave) * 1024u + uint32_t(i) * 4096u);
}

// LDS byte offset of bf16 element (r, c) of a tile.
__device__ inline uint32_t swz_elem(int r, int c) {
  return uint32_t(r * 256 + ((swz_perm(c >> 3) ^ swz_f(r & 15)) << 4) + (c & 7) * 2);
}

__device__ inline bf16x8 lds8(const uint8_t* base, uint32_t off) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(base + off));
}

// MFMA operand (A or B: lane l holds row/column l%32 and k-slots 8*(l/32)+e)
// from a swizzled tile stored k-major: tile row krow(kappa) holds k-slot kappa,
// and the operand's rows/columns are tile columns col0 .. col0+31.  Two
// transposing reads: in every group of 16 lanes, lane i receives element i%4
// of the 8-byte pieces read by lanes i/4 + 4k (k = 0..3), so lane r' of group g
// reads tile row krow(8*hl + 4*h + r'/4), columns col0 + 16g + 4*(r'%4) .. +3.
template <class KRow>
__device__ inline bf16x8 tr_operand(const lds_u8* tile, int col0, int lane, KRow krow) {
  const int rp = lane & 15, g = (lane >> 4) & 1, hl = lane >> 5;
  const int c = col0 + 16 * g + 4 * (rp & 3);
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4i16*)(tile + swz_elem(krow(8 * hl + (rp >> 2)), c)));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4i16*)(tile + swz_elem(krow(8 * hl + 4 + (rp >> 2)), c)));
  const v4i16 v[2] = {lo, hi};
  return __builtin_bit_cast(bf16x8, v);
}

// bf16 B operand for k-step kk (16 rows of a 32-row MFMA result block) from
// the fp32 result registers: rows 16kk + 8j + 4hl + i, j in {0, 1}, i in 0..3,
// i.e. k-slot kappa holds result row 16kk + swap23(kappa).
__device__ inline bf16x8 rows_to_operand(const f32x16& x, int kk) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)x[8 * kk + e];
  return r;
}

// Per-lane parts of operand addresses, computed once per kernel so that every
// read in the loops is a fixed register plus a compile-time offset.
//
// TrTable: transposing reads from a k-major tile whose k-slot kappa of a
// 16-row step starting at row R (a multiple of 16) is row R + kappa
// (natural) or R + swap23(kappa) (SWAP); t[h][cb] is the byte offset, minus
// R*256, of read h of the operand over columns 32*cb .. 32*cb + 31.
struct TrTable {
  uint32_t t[2][4];
};
template <bool SWAP>
__device__ inline TrTable tr_table(int lane) {
  const int rp = lane & 15, g = (lane >> 4) & 1, hl = lane >> 5;
  TrTable T;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int lrow = SWAP ? 8 * h + 4 * hl + (rp >> 2) : 8 * hl + 4 * h + (rp >> 2);
      T.t[h][cb] = swz_elem(lrow, 32 * cb + 16 * g + 4 * (rp & 3));
    }
  return T;
}
__device__ inline bf16x8 tr_op(const lds_u8* tile, const TrTable& T, int R, int cb) {
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(tile + R * 256 + T.t[0][cb]));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(tile + R * 256 + T.t[1][cb]));
  const v4i16 v[2] = {lo, hi};
  return __builtin_bit_cast(bf16x8, v);
}
// RowTable: 16-byte row reads of an A/B operand (lane holds row R + rl, rl = ln
// or swap23(ln), R a multiple of 32; dims 16ks + 8hl .. +7): u[ks] is the
// byte offset minus R*256.
struct RowTable {
  uint32_t u[8];
};
template <bool SWAP>
__device__ inline RowTable row_table(int lane) {
  const int ln = lane & 31, hl = lane >> 5;
  const int rl = SWAP ? swap23(ln) : ln;
  RowTable U;
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) U.u[ks] = swz_elem(rl, 16 * ks + 8 * hl);
  return U;
}
__device__ inline bf16x8 row_op(const uint8_t* tile, const RowTable& U, int R, int ks) {
  return lds8(tile, uint32_t(R * 256) + U.u[ks]);
}

// ---------------------------------------------------------------- dkdv ----

// One workgroup per window key tile kj = ((pos*B + b)*H + h)*NT + t, T/16
// waves (eight for 128-token tiles): wave w < T/32 (group 0) and wave
// w + T/32 (group 1) share keys 32w + swap23(ln) (lane ln), so that the V operand read transposed from the
// pool's V^T tile (whose columns hold the keys in swap23 order) lands in
// natural lane order.  Per 32-query block, group 0 computes S = Q K^T and P,
// hands P (bf16, already in the B-operand layout) to its partner through LDS
// and accumulates dV^T += dO^T P; group 1 computes dP = dO V^T, then
// dS = P (dP - delta) and dK^T += Q^T dS.  The S and dP accumulators start
// from the workspace's -LSE/scale and -delta, so P = exp2(c2 S') and
// dS = P dP' need no subtraction.  Both groups issue the same number of MFMAs
// and one SIMD runs one wave of each.  The kept query tiles are gathered first
// (mask bits); their Q and dO rows are double-buffered in LDS.
__device__ inline uint32_t copy_offset8(int wave, int lane) {
  const int r = 4 * wave + (lane >> 4);
  return uint32_t(r * 256 + swz_perm((lane & 15) ^ swz_f(r & 15)) * 16);
}
// A T-row tile of 256-byte rows with W = T/16 waves: copy i of wave w fills
// LDS chunks [64*(W i + w), +64), rows 4(W i + w) + lane/16; the row's low
// four bits do not depend on i.
template <int W>
__device__ inline void copy_tile_w(const uint8_t* src, uint32_t lds_tile, uint32_t voff, int wave) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    dma16(src + i * (W * 1024), voff, lds_tile + uint32_t(wave) * 1024u + uint32_t(i) * uint32_t(W * 1024));
}
// The V^T of a 64-token page ([128 dims][64 keys], 128-byte rows) into the
// swizzled [128][128] tile layout, of which it fills the first 64 columns,
// with four waves: copy i of wave w fills rows 16i + 4w + lane/16.  A lane
// whose LDS position holds one of the unused columns 64..127 fetches a
// duplicate of a used chunk of its row (in bounds, never read).
__device__ inline uint32_t copy_offset_vt64(int wave, int lane) {
  const int r = 4 * wave + (lane >> 4);
  return uint32_t(r * 128 + (swz_perm((lane & 15) ^ swz_f(r)) & 7) * 16);
}
__device__ inline void copy_vt64_w4(const uint8_t* src, uint32_t lds_tile, uint32_t voff, int wave) {
#pragma unroll
  for (int i = 0; i < 8; ++i) dma16(src + i * 2048, voff, lds_tile + uint32_t(wave) * 1024u + uint32_t(i) * 4096u);
}
__device__ inline uint32_t copy_offset8_page(int wave, int lane) {
  const int r = 4 * wave + (lane >> 4);
  return page_chunk(r, swz_perm((lane & 15) ^ swz_f(r & 15)));
}
__device__ inline void copy_tile8_page(const uint8_t* src, uint32_t lds_tile, uint32_t voff, int wave) {
#pragma unroll
  for (int i = 0; i < 4; ++i) dma16(src + i * 4096, voff, lds_tile + uint32_t(wave) * 1024u + uint32_t(i) * 8192u);
}

template <int T>
__global__ __launch_bounds__(4 * T, 1) void bwd_dkdv_kernel(BwdArgs a) {
  constexpr int kKW = T / 32;                        // key blocks = waves of a group
  constexpr int kQB = T / 32;                        // 32-query blocks of a query tile
  // Q and dO rows, two query tiles (128 KB); the second dO buffer first holds
  // the page's V^T (128 rows)
  __shared__ uint4 sQ[2][kT * 16], sO[2][kT * 16];
  __shared__ uint4 sP[4 * 2 * 2 * 64];               // P operands: [wave pair][block of the half][kk][lane]
  __shared__ float sLD[2][2 * kT];                   // -LSE/scale, then -delta, per buffer
  __shared__ uint16_t sList[kBwdMaxQTiles];
  __shared__ int sN;

  const int kj = blockIdx.x;
  const int t = kj % a.NT;
  const int posbh = kj / a.NT;
  const int bh = posbh % (a.B * a.H);
  const int pos = posbh / (a.B * a.H);
  const int h = bh % a.H, b = bh / a.H;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave / kKW, kw = wave % kKW;
  const int lane = tid & 63, hl = lane >> 5, ln = lane & 31;
  const uint32_t voff = copy_offset8(wave, lane);
  const int kvalid = tile_valid(a.tv, t, a.NT, a.tail, T);
  const int key = kw * 32 + swap23(ln);         // this lane's key (result column)
  const bool key_ok = key < kvalid;
  const int j = pos * a.NT + t;                 // logical key tile
  const uint8_t* qbase = a.work + size_t(bh) * a.NT * kBwdQTile;

  // B operands of the wave's keys: group 0 K rows from the page, group 1 V
  // read transposed from the page's V^T staged in the second dO buffer
  const uint8_t* page = a.pool + ((size_t(a.slot_of[pos]) * a.B * a.H + bh) * a.NT + t) * page_bytes(T, kD);
  bf16x8 bop[8];
  if (grp == 0) {
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const uint32_t off = T == 128 ? page_chunk(key, 2 * ks + hl) : uint32_t(key * 256 + (2 * ks + hl) * 16);
      bop[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(page + off));
    }
  }
  if constexpr (T == 128)
    copy_tile8_page(page + kTile, lds_addr(&sO[1][0]), copy_offset8_page(wave, lane), wave);
  else
    copy_vt64_w4(page + T * kD * 2, lds_addr(&sO[1][0]), copy_offset_vt64(wave, lane), wave);

  // kept query tiles, ascending
  if (wave == 0) {
    int cnt = 0;
    for (int base = 0; base < a.NT; base += 512) {
      uint32_t w[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int i = base + 64 * k + lane;
        w[k] = i < a.NT ? a.mask[size_t(bh * a.NT + i) * a.mask_words + (j >> 5)] : 0u;
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const bool keep = (w[k] >> (j & 31)) & 1u;
        const uint64_t bal = __ballot(keep);
        if (keep) sList[cnt + __popcll(bal & ((uint64_t(1) << lane) - 1))] = uint16_t(base + 64 * k + lane);
        cnt += __popcll(bal);
      }
    }
    if (lane == 0) sN = cnt;
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __syncthreads();
  if (grp == 1) {
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      bop[ks] = tr_operand((const lds_u8*)&sO[1][0], kw * 32, lane, [&](int kap) { return 16 * ks + kap; });
  }
  const int N = __builtin_amdgcn_readfirstlane(sN);
  __syncthreads();                              // V^T consumed: the second buffer is free

  auto record = [&](int n) { return qbase + size_t(__builtin_amdgcn_readfirstlane(int(sList[n]))) * kBwdQTile; };
  auto issue = [&](int n) {
    const uint8_t* rec = record(n);
    copy_tile_w<T / 16>(rec, lds_addr(&sQ[n & 1][0]), voff, wave);
    copy_tile_w<T / 16>(rec + kTile, lds_addr(&sO[n & 1][0]), voff, wave);
    if (wave == 0) dma16(rec + 2 * kTile, uint32_t(lane) * 16u, lds_addr(&sLD[n & 1][0]));
  };

  f32x16 acc[4];                                // dV^T (group 0) or dK^T (group 1): [dim block][32 dims x 32 keys]
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) acc[mb] = f32x16{};
  const float c2 = a.scale_log2;
  uint4* pslot = &sP[(kw * 2 * 2) * 64];        // this wave pair's P operands
  const TrTable TT = tr_table<true>(lane);      // X^T reads: k-slot kappa = query 16kk + swap23(kappa)
  const RowTable RT = row_table<false>(lane);   // X rows: query qb*32 + ln

  // acc^T += X^T op over the block's 32 queries (X = Q or dO rows, read transposed)
  auto accumulate = [&](const lds_u8* x, int qb, const bf16x8 (&op)[2]) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_op(x, TT, qb * 32 + 16 * kk, mb), op[kk], acc[mb], 0, 0, 0);
  };
  // c0 + X K^T (group 0: S - LSE/scale from Q rows) or c0 + X V^T (group 1:
  // dP - delta from dO rows) for 32 queries; c0 holds the per-query term in
  // the result layout (register 4g + e = query qb*32 + 8g + 4hl + e), read
  // from the workspace's per-query values.
  auto product = [&](const uint8_t* x, const float* c, int qb) {
    f32x16 v;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 c4 = *reinterpret_cast<const float4*>(&c[qb * 32 + 8 * g + 4 * hl]);
      v[4 * g] = c4.x;
      v[4 * g + 1] = c4.y;
      v[4 * g + 2] = c4.z;
      v[4 * g + 3] = c4.w;
    }
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      v = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_op(x, RT, qb * 32, ks), bop[ks], v, 0, 0, 0);
    return v;
  };
  // group 0, block qb: S, P (as bf16 B operands, also written to the block's P slot)
  auto scores = [&](const uint8_t* lq, const float* ld, int qb, bf16x8 (&op)[2]) {
    const f32x16 sv = product(lq, ld, qb);      // S - LSE/scale (-inf on padding queries)
    f32x16 p;
#pragma unroll
    for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(sv[r] * c2);
    if (kvalid < T) {                           // padding keys (lanes) weigh nothing
#pragma unroll
      for (int r = 0; r < 16; ++r) p[r] = key_ok ? p[r] : 0.f;
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      op[kk] = rows_to_operand(p, kk);
      pslot[((qb & 1) * 2 + kk) * 64 + lane] = __builtin_bit_cast(uint4, op[kk]);
    }
  };
  // group 1, block qb: dS = P (dP - delta) from the block's P slot, dK^T += Q^T dS
  auto dk_block = [&](const lds_u8* lq, int qb, const f32x16& dpv) {
    f32x16 ds;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      // k-slot e of operand kk is result register 8kk + e
      const bf16x8 pk = __builtin_bit_cast(bf16x8, pslot[((qb & 1) * 2 + kk) * 64 + lane]);
#pragma unroll
      for (int e = 0; e < 8; ++e) ds[8 * kk + e] = float(pk[e]) * dpv[8 * kk + e];
    }
    const bf16x8 op[2] = {rows_to_operand(ds, 0), rows_to_operand(ds, 1)};
    accumulate(lq, qb, op);
  };

  // Per tile, kQB + 1 steps (five for 128-token tiles) separated by
  // meetings; P slot qb&1 carries block qb from group 0 (step qb) to group 1
  // (step qb+1):
  //   step 0:   group 0 S, P of block 0            | group 1 dP of block 0
  //   step s:   group 0 S, P of block s, dV of s-1 | group 1 dS, dK of s-1, dP of s
  //   step kQB: group 0 dV of the last block       | group 1 dS, dK of the last block
  // so that in the middle steps both waves of a SIMD have 16 MFMAs.
  // The buffer of tile n is n&1; the loop runs two tiles per trip so that the
  // buffer, and with it every operand address, is a compile-time offset.
  // Each group runs its own copy of the tile loop (same meetings in the same
  // order), so that no branch on the group sits inside the loop and the
  // accumulators keep their registers.
  auto tile = [&](int n, auto buf, auto group) {
    constexpr int B = decltype(buf)::value;
    constexpr int G = decltype(group)::value;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();                            // tile n in LDS; tile n-1 fully consumed
    if (n + 1 < N) issue(n + 1);
    const uint8_t* lq = reinterpret_cast<const uint8_t*>(&sQ[B][0]);
    const uint8_t* lo = reinterpret_cast<const uint8_t*>(&sO[B][0]);
    const float* ld = &sLD[B][0];
    bf16x8 op[2][2];                            // group 0: P operands of the last two blocks
    f32x16 dpv[2];                              // group 1: dP - delta of the last two blocks
#pragma unroll
    for (int st = 0; st <= kQB; ++st) {
      if constexpr (G == 0) {
        if (st < kQB) scores(lq, ld, st, op[st & 1]);
        if (st > 0) accumulate((const lds_u8*)lo, st - 1, op[(st - 1) & 1]);   // dV^T += dO^T P
      } else {
        if (st > 0) dk_block((const lds_u8*)lq, st - 1, dpv[(st - 1) & 1]);
        if (st < kQB) dpv[st & 1] = product(lo, ld + kT, st);
      }
      if (st < kQB) __syncthreads();            // P of block st written; block st-1 consumed
    }
  };
  auto run = [&](auto group) {
    for (int n = 0; n < N; n += 2) {
      tile(n, std::integral_constant<int, 0>{}, group);
      if (n + 1 < N) tile(n + 1, std::integral_constant<int, 1>{}, group);
    }
  };

  if (N > 0) issue(0);
  if (grp == 0) run(std::integral_constant<int, 0>{});
  else run(std::integral_constant<int, 1>{});

  // store: lane holds key `key`, dims mb*32 + 8*(r/4) + 4*hl + r%4; padding
  // rows inside the chunk (block order) get the zeros they accumulated
  const size_t tok = size_t(t) * T + key;
  if (tok < size_t(a.L)) {
    float* dst = (grp ? a.dk : a.dv) + (((size_t(pos) * a.B + b) * a.L + tok) * a.H + h) * kD;
    const float f = grp ? a.scale : 1.0f;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<float4*>(dst + mb * 32 + 8 * g + 4 * hl) =
            make_float4(acc[mb][4 * g] * f, acc[mb][4 * g + 1] * f, acc[mb][4 * g + 2] * f, acc[mb][4 * g + 3] * f);
  }
}

// ------------------------------------------------------------------ dq ----

// One workgroup per query tile.  The S^T and dP^T result rows of key block kb
// hold keys kb*32 + swap23(m) (m = result row), the order in which the V
// operand arrives when read transposed from the page's V^T; K rows are read
// in the same order.  dS^T as a B operand then holds natural key order.
// Entries naming a tile outside the window count no key.
template <int T>
__global__ __launch_bounds__(2 * T, 2) void bwd_dq_kernel(BwdArgs a) {
  // K rows and V^T of one page in the swizzled 256-byte-row layout (64 KB;
  // a 64-token page fills K's first 64 rows and V^T's first 64 columns)
  __shared__ uint4 sK[kT * 16], sV[kD * 16];

  const int row = blockIdx.x;                  // (b*H + h)*NT + i
  const int i = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H, b = bh / a.H;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, hl = lane >> 5, ln = lane & 31;
  // copy offsets: 128-token pages with four waves, one offset for every copy;
  // 64-token pages with two waves, copy i of wave w filling rows
  // 8i + 4w + lane/16, whose low four bits depend on i % 2
  uint32_t voff = 0, koff64[2] = {0, 0}, voff64[2] = {0, 0};
  if constexpr (T == 128) {
    voff = copy_offset_page(wave, lane);
  } else {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int r = 4 * wave + (lane >> 4) + 8 * k;
      koff64[k] = uint32_t(r * 256 + swz_perm((lane & 15) ^ swz_f(r)) * 16);
      voff64[k] = uint32_t(r * 128 + (swz_perm((lane & 15) ^ swz_f(r)) & 7) * 16);
    }
  }
  const int q = wave * 32 + ln;                 // this lane's query (result column)
  const lds_u8* lk = (const lds_u8*)sK;
  const lds_u8* lv = (const lds_u8*)sV;

  const uint8_t* rec = a.work + size_t(row) * kBwdQTile;
  bf16x8 qf[8], of[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    qf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(rec + size_t(q) * 256 + (2 * ks + hl) * 16));
    of[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(rec + kTile + size_t(q) * 256 + (2 * ks + hl) * 16));
  }
  // per-lane query terms as MFMA seeds: S^T - LSE/scale and dP^T - delta
  const float nl = reinterpret_cast<const float*>(rec + 2 * kTile)[q];
  const float nd = reinterpret_cast<const float*>(rec + 2 * kTile)[kT + q];
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  f32x16 negl, negd;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    negl[r] = nl;
    negd[r] = nd;
  }
  const TrTable TT = tr_table<false>(lane);    // K^T and V reads: k-slot kappa = row R + kappa
  const RowTable RT = row_table<true>(lane);   // K rows kb*32 + swap23(ln)

  f32x16 dqt[4];                                // [4 dim blocks][32 dims x 32 queries]
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) dqt[mb] = f32x16{};
  const float c2 = a.scale_log2;
  const int N = ((const const_i32*)a.counts)[row];
  const const_i32* list = ((const const_i32*)a.idx) + size_t(row) * a.nk_cap;
  const size_t pbytes = page_bytes(T, kD);
  const uint8_t* head_pages = a.pool + size_t(bh) * a.NT * pbytes;
  const size_t slot_stride = size_t(a.B) * a.H * a.NT * pbytes;

  for (int n = 0; n < N; ++n) {
    const int j = list[n];
    int kvalid = 0;
    const uint8_t* page = head_pages + size_t(a.slot_of[0]) * slot_stride;
    if (unsigned(j) < unsigned(a.nk)) {
      const int pos = j / a.NT, t = j - pos * a.NT;
      kvalid = tile_valid(a.tv, t, a.NT, a.tail, T);
      page = head_pages + size_t(a.slot_of[pos]) * slot_stride + size_t(t) * pbytes;
    }
    __syncthreads();                            // previous tile consumed
    if constexpr (T == 128) {
      copy_tile_page(page, lds_addr(sK), voff, wave);
      copy_tile_page(page + kTile, lds_addr(sV), voff, wave);
    } else {
      // K: 64 rows of 256 bytes, 8 copies; V^T: 128 rows of 128 bytes, 16 copies
      const uint32_t lk0 = lds_addr(sK) + uint32_t(wave) * 1024u, lv0 = lds_addr(sV) + uint32_t(wave) * 1024u;
#pragma unroll
      for (int c = 0; c < 8; ++c) dma16(page + (c >> 1) * 4096, koff64[c & 1], lk0 + uint32_t(c) * 2048u);
#pragma unroll
      for (int c = 0; c < 16; ++c)
        dma16(page + T * kD * 2 + (c >> 1) * 2048, voff64[c & 1], lv0 + uint32_t(c) * 2048u);
    }
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
#pragma unroll
    for (int kb = 0; kb < T / 32; ++kb) {
      // S^T = K Q^T and dP^T = V dO^T: A operands are K rows kb*32 + swap23(ln)
      // and V read transposed from V^T (tile row = dim, columns kb*32 ..);
      f32x16 sv, dpv;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        sv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_op((const uint8_t*)sK, RT, kb * 32, ks), qf[ks],
                                                     ks ? sv : negl, 0, 0, 0);
        dpv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_op(lv, TT, 16 * ks, kb), of[ks], ks ? dpv : negd, 0, 0, 0);
      }
      // keys past the tile's valid rows get -inf, so their weights vanish (a
      // rare case: the key indices are formed here, not held across the loop)
      if (kvalid < T) {
        int h4 = 4 * hl;
        asm volatile("" : "+v"(h4));
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kb * 32 + swap23(8 * (r >> 2) + h4 + (r & 3)) >= kvalid) sv[r] = -INFINITY;
      }
      // result row m = 8*(r/4) + 4*hl + r%4 holds key kb*32 + swap23(m)
      f32x16 ds;
#pragma unroll
      for (int r = 0; r < 16; ++r) ds[r] = __builtin_amdgcn_exp2f(sv[r] * c2) * dpv[r];
      // dQ^T += K^T dS^T: k-slot kappa of step kk = key kb*32 + 16kk + kappa
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 db = rows_to_operand(ds, kk);
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
          dqt[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_op(lk, TT, kb * 32 + 16 * kk, mb), db, dqt[mb], 0, 0, 0);
      }
    }
  }

  // padding rows inside the chunk accumulated zeros (their seed is -inf)
  if (size_t(i) * T + q < size_t(a.L)) {
    const size_t base = ((size_t(b) * a.L + size_t(i) * T + q) * a.H + h) * kD;
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

// Scratch of the no-allocation backward: the query-tile records that
// launch_attn_bwd keeps in the caller's workspace, in a file-scope device
// array instead.  Every GPU the library runs on holds its own copy until the
// process ends; in host code the array's name is only a stand-in, so kernels
// are handed its device address, looked up once per device.
static __device__ __align__(256) uint8_t scratch[kBwdScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the device of `stream` (the current device
// for the null stream), looked up with that device current on the first call.
hipError_t scratch_address(hipStream_t stream, void** out) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  int dev = cur;
  if (stream != nullptr && (e = hipStreamGetDevice(stream, &dev)) != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) {
      const hipError_t r = hipSetDevice(cur);
      if (e == hipSuccess) e = r;
    }
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

hipError_t launch_attn_bwd_noalloc(BwdArgs a, hipStream_t stream) {
  if (size_t(a.B) * size_t(a.H) * size_t(a.NT) * kBwdQTile > kBwdScratchBytes) return hipErrorInvalidValue;
  void* p = nullptr;
  hipError_t e = scratch_address(stream, &p);
  if (e != hipSuccess) return e;
  a.work = static_cast<uint8_t*>(p);
  return launch_attn_bwd(a, stream);
}

namespace {

template <int T>
hipError_t launch_bwd_t(const BwdArgs& a, hipStream_t stream) {
  const unsigned qrows = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  const unsigned ktiles = unsigned(a.n_live) * qrows;
  bwd_prep_kernel<T><<<qrows, kThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  bwd_dkdv_kernel<T><<<ktiles, 4 * T, 0, stream>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  bwd_dq_kernel<T><<<qrows, 2 * T, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd(const BwdArgs& a, hipStream_t stream) {
  if (a.T == 128) return launch_bwd_t<128>(a, stream);
  if (a.T == 64) return launch_bwd_t<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace uf
