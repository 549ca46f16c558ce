// attn_fwd (128-token tiles): block-sparse chunk-causal attention forward on
// gfx950 with three wave groups rotating between the matrix core and the
// vector ALU.
//
// For one (b, h, query tile i) the workgroup walks the kept key tiles of its
// list in ascending logical order (Eq. 4: attention restricted to the kept
// blocks of the chunk-causal window) and keeps an online softmax.
//
// Work split.  Twelve waves per workgroup, one workgroup per CU, three waves
// per SIMD: waves w, w+4 and w+8 own the same 32 queries.  The kept tiles are
// cut into units of 64 keys (unit u: tile u/2, key half u%2) and unit u
// belongs to group u%3, which keeps its own running offset, sum and O; the
// three partial states are merged through LDS at the end (log-sum-exp merge).
//
// Rotation.  Phase p (phases separated by workgroup barriers): group p%3
// issues its 32 MFMAs, O^T += V^T P^T of unit p-3 and S^T = K Q^T of unit p,
// while group (p-1)%3 turns the first 32 keys of S(p-1) into weights and
// group (p-2)%3 the last 32 keys of S(p-2).  Each SIMD thus holds one wave on
// the matrix core and two on the vector ALU in every phase: the softmax of a
// unit spans two phases, and two waves issuing VALU work side by side reach
// about twice the issue rate of one.
//
// Products.  K and V^T come from LDS as the A operand, Q^T and P^T are B
// operands in registers, every lane owns one query column (row max and sum
// need one permlane32 exchange), and the weights rounded to bf16 in place are
// the PV operand (V pages keep the keys of each group of 16 in swap23 order,
// the k-slot order of the S^T result lanes).
//
// Memory.  Half tiles (16 KB: 64 keys of K, or 64 keys of V^T with rows d and
// d+64 side by side) are copied HBM -> LDS by global_load_lds, 16 bytes per
// lane.  Copy c of a half tile fills LDS bytes [1 KB c, +1 KB): lane i takes
// 16 bytes of row R = 8(c%8) + i/8, chunk 8(c/8) + (i%8 ^ g(R%16)), where g
// is a 3-bit XOR pattern chosen so that operand reads (16 bytes per lane, 32
// rows) are free of bank conflicts whether 8 or 16 lanes share a cycle; the
// lane's source offset then depends on c only through c%2, and the operand
// read offsets of a lane take four values plus compile-time constants.  The
// pages keep K and V^T in blocks of 64 columns (128-byte rows), so each copy
// reads one contiguous kilobyte: eight consecutive rows of one block.
// Buffers: one K slot per group (K of unit u+3 is copied by group u%3 in its
// first softmax phase, right after the MFMA phase that read K of unit u) and
// six V slots (V of unit u+3 copied in the group's second softmax phase,
// four phases before the PV that reads it); 144 KB in all.  A wave waits for
// its own copies only at the end of its second softmax phase (K of unit u+3
// and, issued before it, V of unit u: both read in the next phase), and the
// barrier after it publishes them to the group.
//
// Softmax in base 2 with a lazy offset m per lane: weights exp2(c2 s - m),
// c2 = scale*log2(e).  The offset is raised only when the weights of a half
// unit sum to more than kSumBound on some lane (or on a lane's first valid
// key); then the exact max is taken, O and l are rescaled, and the weights
// are recomputed (first softmax phase: from the max over the whole unit;
// second: by a whole number of octaves, see tri_second).  The row sum adds
// the fp32 weights before their rounding to bf16: the normalisation then
// differs from the sum of the rounded weights by at most 2^-9 relative, and
// fp32 adds are cheaper here than v_dot2 over the packed weights, which
// slows down next to a stream of MFMAs.
#include "attn_common.h"

#include <type_traits>

namespace uf {
namespace {

using namespace attn;

constexpr int kT = 128;
constexpr int kThreads = 768;          // twelve waves
constexpr uint32_t kHalf = 16384;      // bytes of a half-tile buffer
// LDS buffers of group g: 3g (V slot g), 3g+1 (V slot g+3), 3g+2 (its K slot)
constexpr int kGroupBytes = 3 * kHalf;
constexpr int kBuffers = 9;
constexpr float kSumBound = 4096.0f;   // lane row-sum bound of one half unit's 16 weights
constexpr int kUnitCap = 4095;         // non-empty units of a row listed in LDS

// 3-bit XOR pattern of LDS row r (r % 16): bijective in bits 0..2 for either
// value of bit 3, and in bits 1..3 for either value of bit 0.
__device__ __forceinline__ int swz(int r) {
  const int b3 = (r >> 3) & 1;
  return ((((r >> 2) & 1) ^ b3) << 2) | (r & 2) | ((r & 1) ^ b3);
}

struct TriState {
  f32x16 o[4];     // O^T [4 x 32 dims][32 queries]
  f32x16 s[2];     // raw S^T of the unit's 64 keys (two blocks of 32)
  bf16x8 p[4];     // P^T of the unit: four 16-key steps
  float m;         // offset (base-2 units), -inf until the lane's first valid key
  float moff;      // m, or 0 while m is -inf
  float l;         // this lane's share of the row sum; the partner lane holds the rest
};

// s_waitcnt vmcnt(n) lgkmcnt(0), then the workgroup barrier.  The signal
// fences keep the compiler from moving LDS accesses across the barrier.
template <int N>
__device__ __forceinline__ void sync_vm() {
  constexpr int imm = (N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(imm);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// MFMA phase: O^T += V^T P^T of the previous unit (V^T in the group's buffer
// VB, 0 or 1) and S^T = K Q^T of the current unit (K in the group's buffer 2).
// rg holds the lane's read offsets within the group's 48 KB, so that every
// further offset fits the 16-bit immediate of the LDS instructions.
template <int VB>
__device__ __forceinline__ void tri_mfma(TriState& st, const bf16x8 (&qf)[8], const uint32_t (&rg)[4],
                                         const uint8_t* lds) {
  const uint8_t* vb = lds + VB * kHalf;
  const uint8_t* kb = lds + 2 * kHalf;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const bf16x8 vf = as_bf16x8(*reinterpret_cast<const uint4*>(vb + rg[j] + 4096 * mb));
      st.o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, st.p[j], st.o[mb], 0, 0, 0);
    }
#pragma unroll
  for (int ks = 0; ks < 8; ++ks)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const bf16x8 kf = as_bf16x8(*reinterpret_cast<const uint4*>(kb + rg[ks & 3] + 4096 * h + 8192 * (ks >> 2)));
      st.s[h] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], ks == 0 ? f32x16{} : st.s[h], 0, 0, 0);
    }
  // operand reads: kAhead in flight, then one per MFMA
  constexpr int kReads = 32, kMfma = 32, kAhead = 4;
  __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
  for (int i = 0; i < kReads - kAhead; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, kMfma - (kReads - kAhead), 0);
}

// The four 1-KB copies of a wave for one half tile: copy t is copy c = q + 4t
// of the half tile (q = the wave's query block), source src + 4096 (t % 2) +
// step (t / 2) plus the lane offset, LDS destination lds + 4096 t.
struct HalfCopy {
  const uint8_t* src;
  uint32_t lds;
  uint32_t step;    // source bytes per c/8: the next K block (16384) or the next 64 rows of V^T (8192)
  bool on;
};
// j / NT for 0 <= j < 2^31 from d = (2^64 - 1) / NT: ((j + 1) * d) >> 64 in
// scalar integer arithmetic (a division by a run-time value would otherwise
// use vector float instructions in the softmax waves).  With d = (2^64 - r) / NT,
// 0 < r <= NT, the product is (j + 1) / NT minus less than 2^-32, which floors
// to j / NT.
__device__ __forceinline__ int div_nt(uint32_t j, uint64_t d) {
  const uint64_t x = uint64_t(j) + 1u;
  const uint64_t lo = x * uint32_t(d);
  const uint64_t hi = x * uint32_t(d >> 32);
  return int((hi + (lo >> 32)) >> 32);
}

// A pointer that is the same on every lane, held in scalar registers.
__device__ __forceinline__ const uint8_t* uniform_ptr(const uint8_t* q) {
  const uint64_t p = reinterpret_cast<uint64_t>(q);
  // (the builtin returns int: widen through uint32_t, not by sign extension)
  const uint64_t lo = uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(p)));
  const uint64_t hi = uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(p >> 32)));
  return reinterpret_cast<const uint8_t*>(lo | (hi << 32));
}
__device__ __forceinline__ void half_copy(const HalfCopy& cp, uint32_t lane_off, int t) {
  dma16(uniform_ptr(cp.src + 4096 * (t & 1) + cp.step * (t >> 1)), lane_off, cp.lds + 4096u * uint32_t(t));
}

// Weights of key block H (the lane's 16 scores of keys 32H..32H+31) at the
// current offset into P^T steps 2H, 2H+1; returns the lane's sum of the
// weights (before rounding).  The copies of `cp` are issued along the way.
template <int H, bool COPIES>
__device__ __forceinline__ float tri_weights(TriState& st, float c2, const HalfCopy& cp, uint32_t lane_off) {
  float rs = 0.f;
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    bf16x2 pr[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      // a copy before every second pair of weights, fenced by scheduling
      // barriers (the guarded copies still end up at the start of the phase,
      // but the fences keep the weights in this order, which measured faster)
      if (COPIES && (e & 1) == 0) {
        __builtin_amdgcn_sched_barrier(0);
        if (cp.on) half_copy(cp, lane_off, 2 * jj + (e >> 1));
        __builtin_amdgcn_sched_barrier(0);
      }
      const float x0 = __builtin_fmaf(st.s[H][8 * jj + 2 * e], c2, -st.moff);
      const float x1 = __builtin_fmaf(st.s[H][8 * jj + 2 * e + 1], c2, -st.moff);
      const float w0 = __builtin_amdgcn_exp2f(x0), w1 = __builtin_amdgcn_exp2f(x1);
      pr[e] = bf16x2{(__bf16)w0, (__bf16)w1};
      rs += w0 + w1;
    }
    st.p[2 * H + jj] = __builtin_shufflevector(__builtin_shufflevector(pr[0], pr[1], 0, 1, 2, 3),
                                               __builtin_shufflevector(pr[2], pr[3], 0, 1, 2, 3),
                                               0, 1, 2, 3, 4, 5, 6, 7);
  }
  // Materialise the packed weights here: the rescale that may follow
  // recomputes them, and without this the compiler would keep the unpacked
  // fp32 values alive across it to pack them afterwards.
  asm volatile("" : "+v"(st.p[2 * H]), "+v"(st.p[2 * H + 1]), "+v"(rs));
  return rs;
}

// Keys 32H + 8(e/4) + 4 hl + e%4 of the unit at or past `valid` are padding.
template <int H>
__device__ __forceinline__ void tri_mask(TriState& st, int valid, int hl) {
  if (valid < 64) {
    const int vl = valid - 4 * hl;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const bool pad = H * 32 + 8 * (e >> 2) + (e & 3) >= vl;
      st.s[H][e] = pad ? -INFINITY : st.s[H][e];
    }
  }
}

// The weights of a softmax phase are computed in that phase: an optional
// rescale rewrites them later, which would otherwise let the compiler sink the
// work past the barrier into the next phase.
__device__ __forceinline__ void pin_first(TriState& st) {
  asm volatile("" : "+v"(st.p[0]), "+v"(st.p[1]), "+v"(st.l));
}
__device__ __forceinline__ void pin_second(TriState& st) {
  asm volatile("" : "+v"(st.p[2]), "+v"(st.p[3]), "+v"(st.l));
}

// First softmax phase: padding keys of the unit masked, weights of its first
// 32 keys.  On a lane's first valid key, or when these weights grow too
// large, the offset is set from the exact max over all 64 keys of the unit.
__device__ __forceinline__ void tri_first(TriState& st, int valid, int hl, float c2, const HalfCopy& cp,
                                          uint32_t lane_off) {
  tri_mask<0>(st, valid, hl);
  tri_mask<1>(st, valid, hl);
  float rs0 = tri_weights<0, true>(st, c2, cp, lane_off);
  // wave-uniform: some lane has no offset yet, or its weights grew too large
  if (__ballot(!(st.m > -INFINITY) || rs0 > kSumBound) != 0) {
    float mx = -INFINITY;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, st.s[h][e]);
    mx = pair_max(mx * c2);   // c2 > 0: the max of c2 s over the query's valid keys of the unit
    // Selects, not a per-lane branch: O is rescaled on every lane (by 1 on a
    // lane's first valid key, where O and l are still zero).  The offset
    // stays -inf while the lane has seen no valid key.
    const bool had = st.m > -INFINITY;
    const float sh = had ? fmaxf(mx - st.m, 0.f) : 0.f;
    const float alpha = __builtin_amdgcn_exp2f(-sh);
    st.m = had ? st.m + sh : mx;
    st.l *= alpha;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) st.o[mb] *= alpha;
    st.moff = (st.m > -INFINITY) ? st.m : 0.f;
    rs0 = tri_weights<0, false>(st, c2, cp, lane_off);
  }
  st.l += rs0;
}

// Second softmax phase: weights of the last 32 keys.  When they grow too
// large the offset is raised by a whole number of octaves, so that the first
// half's bf16 weights rescale exactly.  (A lane still without an offset has no
// valid key in the unit: its weights are zero and never trigger this.)
__device__ __forceinline__ void tri_second(TriState& st, float c2, const HalfCopy& cp, uint32_t lane_off) {
  float rs1 = tri_weights<1, true>(st, c2, cp, lane_off);
  if (__ballot(rs1 > kSumBound) != 0) {
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, st.s[1][e]);
    mx = pair_max(mx * c2);
    const float sh = (st.m > -INFINITY) ? ceilf(fmaxf(mx - st.m, 0.f)) : 0.f;
    const float alpha = __builtin_amdgcn_exp2f(-sh);
    st.m += sh;
    st.moff = (st.m > -INFINITY) ? st.m : 0.f;
    st.l *= alpha;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) st.o[mb] *= alpha;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) st.p[j][e] = (__bf16)((float)st.p[j][e] * alpha);
    rs1 = tri_weights<1, false>(st, c2, cp, lane_off);
  }
  st.l += rs1;
}

// SPLIT: the first a.split_from workgroups run rows 0 .. split_from-1 whole;
// each later row r is cut into a.split slices, and workgroup (r, s) takes list
// entries [s*count/split, (s+1)*count/split) of it and writes its unnormalised
// partial (O relative to its offset m, and l) to a.work; a merge combines them.
// UNITS (every window whose rows fit the table, see use_units): the
// workgroup first lists its row's units that hold a valid key (tile j and key
// half, in list order) in LDS and walks only those, so a key half without a
// valid token (block tiles often hold 64 tokens or fewer; a chunk's last tile
// may hold fewer than 65) costs neither copies nor products.
template <bool SPLIT, bool UNITS>
__global__ __launch_bounds__(kThreads, 1) void attn_fwd_tri_kernel(AttnArgs a) {
  __shared__ uint4 sbuf[kBuffers][kHalf / 16];
  __shared__ uint32_t sunit[UNITS ? kUnitCap + 1 : 1];   // (j << 1) | key half; the count last

  int row = int(blockIdx.x), part = 0;
  bool partial = false;               // this workgroup writes a split-KV partial
  if (SPLIT && row >= a.split_from) {
    const int k = row - a.split_from;
    row = a.split_from + k / a.split;
    part = k - (row - a.split_from) * a.split;
    partial = true;
  }
  const int qt = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;          // units u with u % 3 == grp
  const int qw = wave & 3;            // query block of the wave
  const int lane = tid & 63;
  const int hl = lane >> 5;
  const int ln = lane & 31;
  const int qrow = qt * kT + qw * 32 + ln;
  const bool qvalid = qrow < a.L;

  // Q^T as the B operand: lane holds query ln, dims 16*ks + 8*hl .. +8.
  bf16x8 qf[8];
  {
    const uint16_t* qp = a.q + ((size_t(b) * a.L + (qvalid ? qrow : 0)) * a.H + h) * kD + 8 * hl;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      uint4 u = make_uint4(0, 0, 0, 0);
      if (qvalid) u = *reinterpret_cast<const uint4*>(qp + 16 * ks);
      qf[ks] = as_bf16x8(u);
    }
  }
  // Operand read offsets (16-key or 16-dim step j, row ln of a 32-row block)
  // and the lane's copy source offset (copies c with c % 2 == qw % 2).
  uint32_t rd[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) rd[j] = uint32_t(128 * ln + 16 * ((2 * j + hl) ^ swz(ln & 15)));
  const uint32_t lane_off = uint32_t((lane >> 3) * 128 + (((lane & 7) ^ swz(8 * (qw & 1) + (lane >> 3))) * 16));
  const uint8_t* lds = reinterpret_cast<const uint8_t*>(&sbuf[0][0]);
  const uint32_t lds_base = lds_addr(&sbuf[0][0]) + 1024u * uint32_t(qw);

  const size_t pbytes = page_bytes(kT, kD);
  const uint8_t* head_pages = uniform_ptr(a.pool + (size_t(b) * a.H + h) * a.NT * pbytes);
  const size_t slot_stride = size_t(a.B) * a.H * a.NT * pbytes;
  const int total = ((const const_i32*)a.counts)[row];
  const int nsplit = partial ? a.split : 1;
  const int first = partial ? int(int64_t(part) * total / nsplit) : 0;
  const int count = partial ? int(int64_t(part + 1) * total / nsplit) - first : total;
  const float c2 = a.scale_log2;
  const const_i32* list = (const const_i32*)a.idx + size_t(row) * a.nk_cap + first;
  int U = 2 * count;                  // units
  if constexpr (UNITS) {
    // non-empty units of the row's slice, in list order; entries naming a
    // tile outside the window count no key and give none
    // (the list entries of four 64-entry groups are requested together, and
    // their latency overlaps that of the Q loads above)
    if (wave == 0) {
      const int32_t* lv = a.idx + size_t(row) * a.nk_cap + first;
      int off = 0;
      for (int base = 0; base < count; base += 256) {
        uint32_t jj[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int e = base + 64 * k + lane;
          jj[k] = e < count ? uint32_t(lv[e]) : 0xffffffffu;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t j = jj[k];
          int n = 0;
          if (j < uint32_t(a.nk)) {
            const int v = tile_valid(a.tv, int(j % uint32_t(a.NT)), a.NT, a.tail, kT);
            n = (v > 64) ? 2 : (v > 0 ? 1 : 0);
          }
          const uint64_t b1 = __ballot(n >= 1), b2 = __ballot(n == 2);
          const uint64_t below = (uint64_t(1) << lane) - 1;
          const int pos = off + __popcll(b1 & below) + __popcll(b2 & below);
          if (n >= 1) sunit[pos] = j << 1;
          if (n == 2) sunit[pos + 1] = (j << 1) | 1u;
          off += __popcll(b1) + __popcll(b2);
        }
      }
      if (lane == 0) sunit[kUnitCap] = uint32_t(off);
    }
    // Q and the list entries are in registers before any page copy is
    // issued, so that the only vector-memory operations in flight inside the
    // loop are page copies.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    U = int(__builtin_amdgcn_readfirstlane(sunit[kUnitCap]));
  } else {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  }
  const int P = U + 3;                // phases

  // Page and valid keys of unit w (tile w/2, key half w%2).  An entry naming
  // a tile outside the window (stale lists) reads a page of this head and
  // counts no key; units past the list count no key and copy nothing.
  struct Unit {
    const uint8_t* page;
    int valid;
    int half;         // key half of the tile (UNITS; otherwise w % 2)
  };
  auto unit = [&](int w) {
    Unit r{head_pages, 0, 0};
    if (w >= U) return r;
    int j, half;
    if constexpr (UNITS) {
      const uint32_t x = __builtin_amdgcn_readfirstlane(sunit[w]);
      j = int(x >> 1);
      half = int(x & 1u);
    } else {
      j = list[w >> 1];
      half = w & 1;
    }
    r.half = half;
    if (unsigned(j) >= unsigned(a.nk)) {
      r.page = head_pages + size_t(a.slot_of[0]) * slot_stride;
      return r;
    }
    const int pos = div_nt(uint32_t(j), a.nt_div);
    const int t = j - pos * a.NT;
    r.page = head_pages + size_t(a.slot_of[pos]) * slot_stride + size_t(t) * pbytes;
    r.valid = min(max(tile_valid(a.tv, t, a.NT, a.tail, kT) - 64 * half, 0), 64);
    return r;
  };
  // page bytes: K block j (dimensions 64j..) at 16384 j, rows of 128 bytes;
  // V^T block j (keys 64j..) at 32768 + 16384 j.  Copy c of a half: K rows
  // 64(w%2) + 8(c%8) .. of block c/8; V^T rows 8(c%8) + 64(c/8) .. of block w%2.
  auto kcopy = [&](const Unit& un, int w, int kbuf) {
    const int half = UNITS ? un.half : (w & 1);
    return HalfCopy{un.page + 8192 * half + 1024 * qw, lds_base + uint32_t(kbuf) * kHalf, 16384u, w < U};
  };
  auto vcopy = [&](const Unit& un, int w, int vbuf) {
    const int half = UNITS ? un.half : (w & 1);
    return HalfCopy{un.page + 32768 + 16384 * half + 1024 * qw, lds_base + uint32_t(vbuf) * kHalf, 8192u, w < U};
  };
  auto issue = [&](const HalfCopy& cp) {
    if (cp.on)
#pragma unroll
      for (int t = 0; t < 4; ++t) half_copy(cp, lane_off, t);
  };

  TriState st;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
    st.o[mb] = f32x16{};
    st.p[mb] = bf16x8{};
  }
  st.m = -INFINITY;
  st.moff = 0.f;
  st.l = 0.f;

  if (U > 0) {
    // The first PV of each group (unit -3, -2 or -1) multiplies zero weights
    // by V^T buffers 1, 4 and 7 (V slots 3..5), which no copy has filled yet:
    // zero them.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = tid + kThreads * i;   // 0 .. 3071: 1024 uint4 per buffer
      sbuf[3 * (k >> 10) + 1][k & 1023] = make_uint4(0, 0, 0, 0);
    }
    // Each group runs its own copy of the phase sequence (template G); all
    // pass the same P barriers.  Unit u of group G: MFMA phase u, softmax
    // phases u+1 and u+2.  K of unit u lives in buffer 3G+2, V of unit u in
    // V slot u % 6 (buffer 3G, or 3G+1 when u % 6 >= 3).
    auto run = [&](auto Gc) {
      constexpr int G = decltype(Gc)::value;
      // lane read offsets within the group's buffers, kept opaque so that
      // the compiler does not fold the group offset back into immediates too
      // large for the LDS instructions
      uint32_t rg[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        rg[j] = rd[j] + uint32_t(G) * kGroupBytes;
        asm volatile("" : "+v"(rg[j]));
      }
      Unit cur = unit(G);
      // prologue: K of units 0 and 1, V of unit 0; later copies follow the
      // steady-state rule (K[u+3] in phase u+1, V[u+3] in phase u+2)
      if (G == 0) {
        issue(kcopy(cur, 0, 2));
        issue(vcopy(cur, 0, 0));
      }
      if (G == 1) issue(kcopy(cur, 1, 5));
      sync_vm<0>();
      int ph = 0;
      if (G == 1) {   // phase 0, second softmax phase of unit -2: copy V[1]
        issue(vcopy(cur, 1, 3));
        if (1 < U) sync_vm<4>(); else sync_vm<0>();
        ph = 1;
      }
      if (G == 2) {   // phases 0 and 1, softmax phases of unit -1: copy K[2], V[2]
        issue(kcopy(cur, 2, 8));
        sync_vm<63>();
        issue(vcopy(cur, 2, 6));
        if (2 < U) sync_vm<4>(); else sync_vm<0>();
        ph = 2;
      }
      // one cycle of unit u: MFMA, first and second softmax phases.  Q = 0:
      // u % 6 == G (PV reads V slot G+3 and the copy of V[u+3] refills it);
      // Q = 1: u % 6 == G+3 and the other way round.
      auto cycle = [&](auto Qc, int u) -> bool {
        constexpr int Q = decltype(Qc)::value;
        constexpr int VPV = 1 - Q;               // V of unit u-3: the group's buffer VPV
        constexpr int VNEW = 3 * G + VPV;        // V of unit u+3 (same slot, freed by the PV)
        // wave priorities: the MFMA phase first, then the first softmax
        // phase (it issues the K copy), then the second
        __builtin_amdgcn_s_setprio(2);
        tri_mfma<VPV>(st, qf, rg, lds);
        __builtin_amdgcn_s_setprio(1);
        sync_vm<63>();
        if (++ph == P) return false;
        // first softmax phase: K of unit u+3 into buffer G
        const Unit nxt = unit(u + 3);
        const HalfCopy kc = kcopy(nxt, u + 3, 3 * G + 2);
        tri_first(st, cur.valid, hl, c2, kc, lane_off);
        pin_first(st);
        __builtin_amdgcn_s_setprio(0);
        sync_vm<63>();
        if (++ph == P) return false;
        // second softmax phase: V of unit u+3
        const HalfCopy vc = vcopy(nxt, u + 3, VNEW);
        tri_second(st, c2, vc, lane_off);
        pin_second(st);
        if (vc.on) sync_vm<4>(); else sync_vm<0>();
        cur = nxt;
        return ++ph != P;
      };
      for (int u = G;; u += 6) {
        if (!cycle(std::integral_constant<int, 0>{}, u)) break;
        if (!cycle(std::integral_constant<int, 1>{}, u + 3)) break;
      }
    };
    if (grp == 0)
      run(std::integral_constant<int, 0>{});
    else if (grp == 1)
      run(std::integral_constant<int, 1>{});
    else
      run(std::integral_constant<int, 2>{});
  }

  // ---- merge the three key groups: groups 1 and 2 hand (m, l, O) to group 0 ----
  st.l = pair_sum(st.l);
  sync_vm<0>();   // every copy and operand read of the loop is done
  float* xo = reinterpret_cast<float*>(&sbuf[0][0]);                    // [8 waves][4][16][64 lanes]: 128 KB
  float* xm = reinterpret_cast<float*>(&sbuf[0][0]) + 8 * 4 * 16 * 64;  // [2][8 waves][64 lanes]: m, then l
  if (grp != 0) {
    const int w = (grp - 1) * 4 + qw;
    xm[w * 64 + lane] = st.m;
    xm[512 + w * 64 + lane] = st.l;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) xo[((w * 4 + mb) * 16 + e) * 64 + lane] = st.o[mb][e];
  }
  sync_vm<0>();
  if (grp == 0) {
    const int w1 = qw, w2 = 4 + qw;
    const float mB = xm[w1 * 64 + lane], lB = xm[512 + w1 * 64 + lane];
    const float mC = xm[w2 * 64 + lane], lC = xm[512 + w2 * 64 + lane];
    const float mm = fmaxf(fmaxf(st.m, mB), mC);
    const float fa = (st.m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(st.m - mm);
    const float fb = (mB == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mB - mm);
    const float fc = (mC == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mC - mm);
    const float l = st.l * fa + lB * fb + lC * fc;
    auto merged = [&](int mb, int e) {
      return st.o[mb][e] * fa + xo[((w1 * 4 + mb) * 16 + e) * 64 + lane] * fb +
             xo[((w2 * 4 + mb) * 16 + e) * 64 + lane] * fc;
    };
    if (SPLIT && partial) {
      if (qvalid) {
        const size_t wrow = size_t(row - a.split_from) * a.split + part;
        float* op = a.work + (wrow * kT + qw * 32 + ln) * kD;
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int d0 = mb * 32 + 8 * i + 4 * hl;
            float4 v;
            v.x = merged(mb, 4 * i + 0);
            v.y = merged(mb, 4 * i + 1);
            v.z = merged(mb, 4 * i + 2);
            v.w = merged(mb, 4 * i + 3);
            *reinterpret_cast<float4*>(op + d0) = v;
          }
        if (hl == 0) {
          const size_t wrows = (size_t(a.B) * a.H * a.NT - a.split_from) * a.split;
          float2* ml = reinterpret_cast<float2*>(a.work + wrows * kT * kD);
          ml[wrow * kT + qw * 32 + ln] = make_float2(mm, l);
        }
      }
      return;
    }
    if (qvalid) {
      const float inv = (l > 0.f) ? 1.f / l : 0.f;
      uint16_t* op = a.o + ((size_t(b) * a.L + qrow) * a.H + h) * kD;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d0 = mb * 32 + 8 * i + 4 * hl;
          uint2 w;
          w.x = pack_bf16x2(merged(mb, 4 * i + 0) * inv, merged(mb, 4 * i + 1) * inv);
          w.y = pack_bf16x2(merged(mb, 4 * i + 2) * inv, merged(mb, 4 * i + 3) * inv);
          *reinterpret_cast<uint2*>(op + d0) = w;
        }
      if (a.lse != nullptr && hl == 0)
        a.lse[(size_t(b) * a.H + h) * a.L + qrow] = (l > 0.f) ? (mm + log2f(l)) * 0.69314718055994531f : -INFINITY;
    }
  }
}

// Split-KV merge (tiles of TT tokens): one workgroup per split row; lane (query, half) combines the
// row's partials for 64 dims: O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.
template <int TT>
__global__ __launch_bounds__(2 * TT) void attn_split_merge_kernel(AttnArgs a) {
  const int row = a.split_from + int(blockIdx.x);
  const int qt = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int ql = threadIdx.x >> 1;
  const int half = threadIdx.x & 1;
  const int qrow = qt * TT + ql;
  if (qrow >= a.L) return;
  const size_t wrows = (size_t(a.B) * a.H * a.NT - a.split_from) * a.split;
  const float2* ml = reinterpret_cast<const float2*>(a.work + wrows * TT * kD);
  float mm = -INFINITY;
  for (int s = 0; s < a.split; ++s) {
    const float2 v = ml[(size_t(row - a.split_from) * a.split + s) * TT + ql];
    if (v.y > 0.f) mm = fmaxf(mm, v.x);
  }
  float acc[64];
#pragma unroll
  for (int d = 0; d < 64; ++d) acc[d] = 0.f;
  float l = 0.f;
  for (int s = 0; s < a.split; ++s) {
    const size_t wrow = size_t(row - a.split_from) * a.split + s;
    const float2 v = ml[wrow * TT + ql];
    if (!(v.y > 0.f)) continue;   // empty slice
    const float w = __builtin_amdgcn_exp2f(v.x - mm);
    l += v.y * w;
    const float4* op = reinterpret_cast<const float4*>(a.work + (wrow * TT + ql) * kD + 64 * half);
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const float4 o = op[c];
      acc[4 * c + 0] += o.x * w;
      acc[4 * c + 1] += o.y * w;
      acc[4 * c + 2] += o.z * w;
      acc[4 * c + 3] += o.w * w;
    }
  }
  const float inv = (l > 0.f) ? 1.f / l : 0.f;
  uint16_t* out = a.o + ((size_t(b) * a.L + qrow) * a.H + h) * kD + 64 * half;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    uint4 w;
    w.x = pack_bf16x2(acc[8 * c + 0] * inv, acc[8 * c + 1] * inv);
    w.y = pack_bf16x2(acc[8 * c + 2] * inv, acc[8 * c + 3] * inv);
    w.z = pack_bf16x2(acc[8 * c + 4] * inv, acc[8 * c + 5] * inv);
    w.w = pack_bf16x2(acc[8 * c + 6] * inv, acc[8 * c + 7] * inv);
    reinterpret_cast<uint4*>(out)[c] = w;
  }
  if (a.lse != nullptr && half == 0)
    a.lse[(size_t(b) * a.H + h) * a.L + qrow] = (l > 0.f) ? (mm + log2f(l)) * 0.69314718055994531f : -INFINITY;
}

}  // namespace

// The unit table holds every unit of a row when 2 * nk_cap <= kUnitCap (windows
// of up to 2,047 key tiles).  It pays on raster windows as well (1K and 2K 1 %
// faster than walking the list with scalar loads: the walk reads one LDS word
// per unit, and the empty second half of a chunk's last tile is skipped).
inline bool use_units(const AttnArgs& a) { return 2 * a.nk_cap <= kUnitCap; }

hipError_t launch_attn_fwd_t128_tri(const AttnArgs& a, hipStream_t stream) {
  const unsigned blocks = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  if (use_units(a))
    attn_fwd_tri_kernel<false, true><<<blocks, kThreads, 0, stream>>>(a);
  else
    attn_fwd_tri_kernel<false, false><<<blocks, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_attn_fwd_t128_tri_split(const AttnArgs& a, hipStream_t stream) {
  const unsigned rows = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  const unsigned blocks = unsigned(a.split_from) + (rows - unsigned(a.split_from)) * unsigned(a.split);
  if (use_units(a))
    attn_fwd_tri_kernel<true, true><<<blocks, kThreads, 0, stream>>>(a);
  else
    attn_fwd_tri_kernel<true, false><<<blocks, kThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_attn_split_merge(a, stream);
}

hipError_t launch_attn_split_merge(const AttnArgs& a, hipStream_t stream) {
  const unsigned rows = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT) - unsigned(a.split_from);
  if (rows == 0) return hipSuccess;
  if (a.T == 128)
    attn_split_merge_kernel<128><<<rows, 256, 0, stream>>>(a);
  else
    attn_split_merge_kernel<64><<<rows, 128, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
