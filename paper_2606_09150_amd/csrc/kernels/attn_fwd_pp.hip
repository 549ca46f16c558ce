// attn_fwd (128-token tiles): block-sparse chunk-causal attention forward on
// gfx950 with a key-split ping-pong between two wave groups.
//
// For one (b, h, query tile i) the workgroup walks the kept key tiles of its
// list in ascending logical order (Eq. 4: attention restricted to the kept
// blocks of the chunk-causal window) and keeps an online softmax.
//
// Work split.  Eight waves per workgroup, one workgroup per CU, two waves per
// SIMD.  Waves w and w+4 own the same 32 queries; group A (waves 0-3) takes
// keys 0..63 of every kept tile, group B (waves 4-7) keys 64..127, each with
// its own running max, sum and O.  The two partial states are merged through
// LDS at the end (flash-decoding style log-sum-exp merge).
//
// Ping-pong.  Per tile there are two phases separated by workgroup barriers.
// In one phase group A issues its MFMA work (PV of the previous tile, S of the
// current one) while group B runs its softmax VALU work, in the next phase the
// roles swap; the two waves sharing a SIMD therefore alternate between the
// matrix core and the vector ALU instead of contending for one of them.
//
// Products.  S^T = K Q^T and O^T += V^T P^T on v_mfma_f32_32x32x16_bf16: K and
// V^T come from LDS as the A operand, Q^T and P^T are B operands held in
// registers; every lane owns one query column, so the row max and row sum
// need one exchange with the partner lane (permlane32 swap), and the
// exponentiated scores are rounded to bf16 in place to serve as the PV operand
// (V pages store the keys of each group of 16 in swap23 order, which is the
// k-slot order of the S^T result lanes).
//
// Memory.  Whole tiles are copied HBM -> LDS by direct global_load_lds
// (16 bytes per lane, XOR-swizzled 16-byte chunks, conflict-free operand
// reads) into two K and three V tile buffers (160 KB, all of the CU's LDS).
// The copies are issued by the group that is in its softmax phase, spread
// through its VALU work (which has slack against the other group's MFMA
// phase), so the MFMA phases carry no copy instructions and the per-CU memory
// pipeline is fed evenly: group B requests K tile m+1 during phase 2m (first
// read at phase 2m+2), group A requests V tile m+1 during phase 2m+1 (first
// read at phase 2m+4).  A buffer is refilled only after a barrier that
// follows its last read.
//
// Softmax in base 2.  Every S accumulator starts at -m / (scale*log2(e)),
// where m is the lane's current offset in base-2 units, so a weight costs one
// multiply and one exp2.  The offset is not the exact running max: it is
// raised only when the weights it gives grow too large, which the row sums
// (bf16-rounded weights added with v_dot2_f32_bf16) reveal without a max
// reduction.  Then, and on a lane's first valid key, the exact max is taken,
// O and l are rescaled and the tile's weights are recomputed (a weight that
// overflowed to inf against a stale offset shows up in the sum as well).
// Weights stay below 2^12 before normalisation, far from overflow, and the
// normalisation by l makes the result independent of the offset up to
// rounding.
#include "attn_common.h"

#include <type_traits>

namespace uf {
namespace {

using namespace attn;

constexpr int kT = 128;
constexpr int kThreads = 512;                 // eight waves
constexpr uint32_t kTileLds = kT * kD * 2;    // 32 KB per K or V tile buffer

struct PPState {
  f32x16 o[4];       // O^T [4 x 32 dims][32 queries]
  // c2 = scale * log2(e)
  f32x16 s[2];       // S^T - m/c2 of the group's 64 keys of the current tile (raw score units)
  bf16x8 p[4];       // P^T operands of the previous tile: four 16-key steps
  f32x16 negm;       // -m/c2 broadcast (0 while m is -inf): initial value of S accumulators
  float m;           // offset (base-2 units), -inf until the lane's first valid key
  float l;           // this lane's share of the row sum; the partner lane holds the rest
};

// Row-sum bound of one lane's 32 weights above which the offset is raised.
constexpr float kSumBound = 4096.0f;

// MFMA phase of group G: PV of the previous tile (buffer pbuf) and S of the
// current tile (buffer sbuf).
template <int G, bool DO_PV, bool DO_S>
__device__ __forceinline__ void pp_mfma(PPState& st, const bf16x8 (&qf)[8], const uint32_t (&rd)[8],
                                        const uint8_t* lds_k, const uint8_t* lds_v, int pbuf, int sbuf) {
  if constexpr (DO_PV) {
    const uint8_t* vbase = lds_v + pbuf * kTileLds;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const bf16x8 vf = as_bf16x8(*reinterpret_cast<const uint4*>(vbase + rd[4 * G + j] + mb * 8192));
        st.o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, st.p[j], st.o[mb], 0, 0, 0);
      }
  }
  if constexpr (DO_S) {
    const uint8_t* kbase = lds_k + sbuf * kTileLds + G * 64 * 256;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 kf = as_bf16x8(*reinterpret_cast<const uint4*>(kbase + rd[ks] + kb * 8192));
        st.s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], ks == 0 ? st.negm : st.s[kb], 0, 0, 0);
      }
  }
  // Keep a bounded number of operand reads in flight: six ahead, then one
  // read per MFMA (bounds register use; hides LDS latency).
  constexpr int kN = (DO_PV ? 16 : 0) + (DO_S ? 16 : 0);
  constexpr int kAhead = 6;
  __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
  for (int i = 0; i < kN - kAhead; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, kAhead, 0);
}

// Copies issued during a softmax phase: eight 16-byte-per-lane copies of the
// wave (copy i fills chunks [64*(4i + q), +64) of the target tile buffer).
struct CopyJob {
  const uint8_t* src;   // uniform page block
  uint32_t lds;         // LDS byte address of the target buffer plus 1 KB * q
  bool on;
};

// Weights exp2(s - sh) of the group's 64 keys as P^T operands; returns the
// lane's sum of the bf16-rounded weights.  The copies of `cj` are spread
// through the work when `copies` is set.
template <bool SHIFT>
__device__ __forceinline__ float pp_weights(PPState& st, float c2, float sh, const CopyJob& cj, const uint32_t (&dma)[8],
                                            bool copies) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float rs = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int kb = j >> 1, hh = j & 1;
    if (copies && cj.on) {
      dma16(cj.src, dma[2 * j], cj.lds + uint32_t(2 * j) * 4096u);
      dma16(cj.src, dma[2 * j + 1], cj.lds + uint32_t(2 * j + 1) * 4096u);
    }
    bf16x2 pr[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float x0 = st.s[kb][8 * hh + 2 * e] * c2, x1 = st.s[kb][8 * hh + 2 * e + 1] * c2;
      if constexpr (SHIFT) {
        x0 -= sh;
        x1 -= sh;
      }
      pr[e] = bf16x2{(__bf16)__builtin_amdgcn_exp2f(x0), (__bf16)__builtin_amdgcn_exp2f(x1)};
      rs = __builtin_amdgcn_fdot2_f32_bf16(pr[e], ones, rs, false);
    }
    st.p[j] = __builtin_shufflevector(__builtin_shufflevector(pr[0], pr[1], 0, 1, 2, 3),
                                      __builtin_shufflevector(pr[2], pr[3], 0, 1, 2, 3),
                                      0, 1, 2, 3, 4, 5, 6, 7);
  }
  return rs;
}

// VALU phase: weights of the group's 64 keys of the current tile; `valid` is
// the number of valid keys among them (0..64).
__device__ __forceinline__ void pp_softmax(PPState& st, int valid, int hl, float c2, const CopyJob& cj,
                                           const uint32_t (&dma)[8]) {
  if (valid < 64) {
    // key kb*32 + 8*(e>>2) + 4*hl + (e&3) is padding when it is >= valid
    const int vl = valid - 4 * hl;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (kb * 32 + 8 * (e >> 2) + (e & 3) >= vl) st.s[kb][e] = -INFINITY;
  }
  float rs = pp_weights<false>(st, c2, 0.f, cj, dma, true);
  // wave-uniform: some lane has no offset yet, or its weights grew too large
  if (__ballot(!(st.m > -INFINITY) || rs > kSumBound) != 0) {
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, st.s[kb][e] * c2);
    mx = pair_max(mx);   // max of c2 * s - m over the query's valid keys of this tile
    float sh;
    if (st.m > -INFINITY) {
      sh = fmaxf(mx, 0.f);
      const float alpha = __builtin_amdgcn_exp2f(-sh);
      st.m += sh;
      st.l *= alpha;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) st.o[mb] *= alpha;
    } else {
      // first valid key of the lane (s holds the raw exponents): offset = max
      sh = (mx > -INFINITY) ? mx : 0.f;
      st.m = mx;
    }
    const float nm = (st.m > -INFINITY) ? -st.m / c2 : 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) st.negm[e] = nm;
    rs = pp_weights<true>(st, c2, sh, cj, dma, false);
  }
  st.l += rs;
}

// SPLIT: workgroup (row, s) of a split-KV launch takes list entries
// [s*count/split, (s+1)*count/split) of its row and writes its unnormalised
// partial (O relative to its offset m, and l) to a.work; a merge combines them.
template <bool SPLIT>
__global__ __launch_bounds__(kThreads, 1) void attn_fwd_pp_kernel(AttnArgs a) {
  __shared__ uint4 sK[2][kT * 16];   // two K tiles: 128 key rows x 16 chunks
  __shared__ uint4 sV[3][kD * 16];   // three V^T tiles: 128 dim rows x 16 chunks

  const int row = SPLIT ? int(blockIdx.x) / a.split : int(blockIdx.x);
  const int part = SPLIT ? int(blockIdx.x) - row * a.split : 0;
  const int qt = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;          // 0: keys 0..63, 1: keys 64..127
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
      const bf16x8 raw = as_bf16x8(u);
      qf[ks] = raw;
    }
  }
  // Q is in registers before any page copy is issued, so that the only
  // vector-memory operations in flight inside the loop are page copies.
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));

  // Copy i of wave q of a group fills LDS chunks [64*(4i + q), +64) of a tile buffer; row
  // r chunk c is stored at r*16 + (c ^ (r & 15)) (K rows = keys, V^T rows =
  // dims).  Operand reads: row ln of a 32-row block, logical chunk 2j + hl.
  uint32_t dma[8], rd[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int p = (4 * i + qw) * 64 + lane;
    const int r = p >> 4, cs = p & 15;
    dma[i] = uint32_t(r * 256 + ((cs ^ (r & 15)) * 16));
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) rd[j] = uint32_t(ln * 256 + (((2 * j + hl) ^ (ln & 15)) * 16));
  const uint32_t k_lds = lds_addr(&sK[0][0]) + uint32_t(qw) * 1024u;
  const uint32_t v_lds = lds_addr(&sV[0][0]) + uint32_t(qw) * 1024u;
  const uint8_t* lds_k = reinterpret_cast<const uint8_t*>(&sK[0][0]);
  const uint8_t* lds_v = reinterpret_cast<const uint8_t*>(&sV[0][0]);

  const size_t pbytes = page_bytes(kT, kD);
  const uint8_t* head_pages = a.pool + (size_t(b) * a.H + h) * a.NT * pbytes;
  const size_t slot_stride = size_t(a.B) * a.H * a.NT * pbytes;
  const int total = ((const const_i32*)a.counts)[row];
  const int first = SPLIT ? int(int64_t(part) * total / a.split) : 0;
  const int count = SPLIT ? int(int64_t(part + 1) * total / a.split) - first : total;
  const float c2 = a.scale_log2;
  const int N = count;
  const const_i32* list = (const const_i32*)a.idx + size_t(row) * a.nk_cap + first;

  // Page of list entry n and its valid keys.  An entry naming a tile outside
  // the window (stale lists) reads a page of this head and counts no key.
  auto page_of = [&](int n, int& valid) {
    const int j = list[n];
    if (unsigned(j) >= unsigned(a.nk)) {
      valid = 0;
      return head_pages + size_t(a.slot_of[0]) * slot_stride;
    }
    const int pos = j / a.NT;
    const int t = j - pos * a.NT;
    valid = tile_valid(a.tv, t, a.NT, a.tail, kT);
    return head_pages + size_t(a.slot_of[pos]) * slot_stride + size_t(t) * pbytes;
  };
  // Copy jobs: K tile n into K buffer n % 2, V tile n into V buffer n % 3.
  auto kjob = [&](int n) {
    CopyJob c;
    c.on = n < N;
    int v;
    c.src = c.on ? page_of(n, v) : head_pages;
    c.lds = k_lds + uint32_t(n & 1) * kTileLds;
    return c;
  };
  auto vjob = [&](int n) {
    CopyJob c;
    c.on = n < N;
    int v;
    c.src = (c.on ? page_of(n, v) : head_pages) + size_t(kT) * kD * 2;
    c.lds = v_lds + uint32_t(n % 3) * kTileLds;
    return c;
  };
  auto issue = [&](const CopyJob& c) {
#pragma unroll
    for (int i = 0; i < 8; ++i) dma16(c.src, dma[i], c.lds + uint32_t(i) * 4096u);
  };
  auto group_valid = [&](int n) {
    int v;
    page_of(n, v);
    return min(max(v - 64 * grp, 0), 64);
  };
  auto sync = [&]() {
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_barrier();
  };

  PPState st;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) st.o[mb] = f32x16{};
  st.negm = f32x16{};
  st.m = -INFINITY;
  st.l = 0.f;

  if (N > 0) {
    // prologue: B copies K tile 0 (needed by phase 0), A copies V tile 0
    if (grp == 1) {
      issue(kjob(0));
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    } else {
      issue(vjob(0));
    }
    __builtin_amdgcn_s_barrier();

    // Phase pair m: phase 2m (A: MFMA, B: softmax), phase 2m+1 (A: softmax,
    // B: MFMA).  m = 0 and m = N are peeled so that the steady-state body is
    // a single variant.  Each group runs its own copy of the phase sequence;
    // both copies pass the same barriers in the same order.
    // top(m): barrier ahead of phase 2m.  B's K tile m (copied in phase
    // 2m-2) has landed; A's V tile m-1 (copied in phase 2m-3) has landed
    // while its V tile m (copied in phase 2m-1) may still be in flight.
    auto top = [&](int m) {
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      if (grp == 0 && m < N)
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(8));
      else
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
      __builtin_amdgcn_s_barrier();
    };
    const CopyJob none = {head_pages, 0u, false};
    auto mfma_phase = [&](auto G, auto do_pv, auto do_s, int m) {
      __builtin_amdgcn_s_setprio(1);
      pp_mfma<decltype(G)::value, decltype(do_pv)::value, decltype(do_s)::value>(
          st, qf, rd, lds_k, lds_v, (m + 2) % 3, m & 1);
      __builtin_amdgcn_s_setprio(0);
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using T = std::true_type;
    using F = std::false_type;
    if (grp == 0) {
      mfma_phase(I0{}, F{}, T{}, 0);
      sync();
      pp_softmax(st, group_valid(0), hl, c2, vjob(1), dma);
      for (int m = 1; m < N; ++m) {
        top(m);
        mfma_phase(I0{}, T{}, T{}, m);
        sync();
        pp_softmax(st, group_valid(m), hl, c2, vjob(m + 1), dma);
      }
      top(N);
      mfma_phase(I0{}, T{}, F{}, N);
      sync();
    } else {
      issue(kjob(1));   // phase 0: B has no softmax work yet
      sync();
      mfma_phase(I1{}, F{}, T{}, 0);
      for (int m = 1; m < N; ++m) {
        top(m);
        pp_softmax(st, group_valid(m - 1), hl, c2, kjob(m + 1), dma);
        sync();
        mfma_phase(I1{}, T{}, T{}, m);
      }
      top(N);
      pp_softmax(st, group_valid(N - 1), hl, c2, none, dma);
      sync();
      mfma_phase(I1{}, T{}, F{}, N);
    }
  }

  // ---- merge the two key halves: group B hands (m, l, O) to group A ----
  st.l = pair_sum(st.l);
  sync();   // every operand read of the loop is done; the K buffers are free
  float* xo = reinterpret_cast<float*>(&sK[0][0]);   // [4 waves][4 blocks][16][64 lanes]: 64 KB
  float* xm = reinterpret_cast<float*>(&sV[0][0]);   // [2][4 waves][64 lanes]: m, then l (V buffer 0)
  if (grp == 1) {
    xm[qw * 64 + lane] = st.m;
    xm[256 + qw * 64 + lane] = st.l;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) xo[((qw * 4 + mb) * 16 + e) * 64 + lane] = st.o[mb][e];
  }
  sync();
  if (grp == 0) {
    const float mB = xm[qw * 64 + lane];
    const float lB = xm[256 + qw * 64 + lane];
    const float mm = fmaxf(st.m, mB);
    const float fa = (st.m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(st.m - mm);
    const float fb = (mB == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mB - mm);
    const float l = st.l * fa + lB * fb;
    if (SPLIT) {
      if (qvalid) {
        const size_t wrow = size_t(row) * a.split + part;
        float* op = a.work + (wrow * kT + qw * 32 + ln) * kD;
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int d0 = mb * 32 + 8 * i + 4 * hl;
            float4 v;
            v.x = st.o[mb][4 * i + 0] * fa + xo[((qw * 4 + mb) * 16 + 4 * i + 0) * 64 + lane] * fb;
            v.y = st.o[mb][4 * i + 1] * fa + xo[((qw * 4 + mb) * 16 + 4 * i + 1) * 64 + lane] * fb;
            v.z = st.o[mb][4 * i + 2] * fa + xo[((qw * 4 + mb) * 16 + 4 * i + 2) * 64 + lane] * fb;
            v.w = st.o[mb][4 * i + 3] * fa + xo[((qw * 4 + mb) * 16 + 4 * i + 3) * 64 + lane] * fb;
            *reinterpret_cast<float4*>(op + d0) = v;
          }
        if (hl == 0) {
          float2* ml = reinterpret_cast<float2*>(a.work + size_t(a.B) * a.H * a.NT * a.split * kT * kD);
          ml[wrow * kT + qw * 32 + ln] = make_float2(mm, l);
        }
      }
      return;
    }
    if (qvalid) {
      const float inv = (l > 0.f) ? 1.f / l : 0.f;
      const float wa = fa * inv, wb = fb * inv;
      uint16_t* op = a.o + ((size_t(b) * a.L + qrow) * a.H + h) * kD;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d0 = mb * 32 + 8 * i + 4 * hl;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            v[e] = st.o[mb][4 * i + e] * wa + xo[((qw * 4 + mb) * 16 + 4 * i + e) * 64 + lane] * wb;
          uint2 w;
          w.x = pack_bf16x2(v[0], v[1]);
          w.y = pack_bf16x2(v[2], v[3]);
          *reinterpret_cast<uint2*>(op + d0) = w;
        }
      if (a.lse != nullptr && hl == 0)
        a.lse[(size_t(b) * a.H + h) * a.L + qrow] = (l > 0.f) ? (mm + log2f(l)) * 0.69314718055994531f : -INFINITY;
    }
  }
}

// Split-KV merge: one workgroup per row; lane (query, half) combines the
// row's partials for 64 dims: O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.
__global__ __launch_bounds__(256) void attn_split_merge_kernel(AttnArgs a) {
  const int row = blockIdx.x;
  const int qt = row % a.NT;
  const int bh = row / a.NT;
  const int h = bh % a.H;
  const int b = bh / a.H;
  const int ql = threadIdx.x >> 1;
  const int half = threadIdx.x & 1;
  const int qrow = qt * kT + ql;
  if (qrow >= a.L) return;
  const float2* ml = reinterpret_cast<const float2*>(a.work + size_t(a.B) * a.H * a.NT * a.split * kT * kD);
  float mm = -INFINITY;
  for (int s = 0; s < a.split; ++s) {
    const float2 v = ml[(size_t(row) * a.split + s) * kT + ql];
    if (v.y > 0.f) mm = fmaxf(mm, v.x);
  }
  float acc[64];
#pragma unroll
  for (int d = 0; d < 64; ++d) acc[d] = 0.f;
  float l = 0.f;
  for (int s = 0; s < a.split; ++s) {
    const size_t wrow = size_t(row) * a.split + s;
    const float2 v = ml[wrow * kT + ql];
    if (!(v.y > 0.f)) continue;   // empty slice
    const float w = __builtin_amdgcn_exp2f(v.x - mm);
    l += v.y * w;
    const float4* op = reinterpret_cast<const float4*>(a.work + (wrow * kT + ql) * kD + 64 * half);
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

hipError_t launch_attn_fwd_t128_pp(const AttnArgs& a, hipStream_t stream) {
  const unsigned blocks = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  attn_fwd_pp_kernel<false><<<blocks, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_attn_fwd_t128_pp_split(const AttnArgs& a, hipStream_t stream) {
  const unsigned rows = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  attn_fwd_pp_kernel<true><<<rows * unsigned(a.split), kThreads, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_attn_split_merge(a, stream);
}

hipError_t launch_attn_split_merge(const AttnArgs& a, hipStream_t stream) {
  const unsigned rows = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  attn_split_merge_kernel<<<rows, 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace uf
