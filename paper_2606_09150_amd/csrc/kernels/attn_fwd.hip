// attn_fwd (64-token tiles): block-sparse chunk-causal attention forward on
// gfx950.
//
// For one (b, h, query tile i) the workgroup walks the kept key tiles of its
// list (Eq. 4: attention restricted to the kept blocks of the chunk-causal
// window) and keeps an online softmax.
//
// Work split: four waves, two key groups of two.  Wave (g, w) holds queries
// 32w .. 32w+31 of the tile and walks list entries g, g + 2, g + 4, ...; each
// group keeps its own (m, l, O), and at the end group 1 hands its state to
// group 0 through LDS (log-sum-exp merge).  A row's walk is a chain of
// dependent steps (copy, S, softmax, PV) with one wave per SIMD, so two groups
// halve its length.  The kernel computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (K from LDS as the A operand, Q held in registers as
// the B operand), so in the result layout every lane owns one query column and
// 16 key rows per 32-key block; the row max and row sum need one exchange with
// the partner lane (permlane32 swap).  The exponentiated scores are rounded to
// bf16 in place and reused directly as the B operand of O^T += V^T P^T; V pages
// are stored transposed with the keys of each group of 16 in swap23 order,
// which is exactly the k-slot order in which the S^T result lanes hold them.
//
// Memory pipeline: pages are copied HBM -> LDS by direct global_load_lds
// (16 bytes per lane, no register staging) into one K buffer and one V buffer
// per group with an XOR swizzle of 16-byte chunks (conflict-free MFMA operand
// reads).  A group requests K of its next tile as soon as every wave has read
// the current K (so it lands during softmax and PV), and V of its next tile as
// soon as every wave has read the current V (so it lands during the next S).
// Both groups run the same number of steps (a group without a tile in a step
// idles through it), so the workgroup barriers that publish the copies match.
//
// Softmax runs in base 2 with scale*log2(e) folded into one FMA.  The running
// max is raised lazily: O and l are rescaled only when some lane's tile max
// exceeds its running max by more than 8 (base-2 units), so exponentials stay
// <= 2^8 and the rescale is rare.  Row sums add the bf16-rounded weights that
// the PV product uses (v_dot2_f32_bf16).  O is normalised once at the end and
// rounded to bf16 (nearest even).
#include "attn_common.h"

namespace uf {
namespace {

using namespace attn;

// With one wave per SIMD nothing hides an operand read's LDS latency but the
// wave's own MFMAs: keep kAhead reads in flight, then one read per MFMA.
template <int kReads>
__device__ inline void schedule_reads_ahead() {
  constexpr int kAhead = 8;
  __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
  for (int i = 0; i < kReads - kAhead; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, kAhead, 0);
}

// SPLIT: as in the 128-token kernel, the first a.split_from workgroups run
// rows 0 .. split_from-1 whole and every later row is cut into a.split slices
// of its list; a slice writes its unnormalised O, its offset (base-2 units)
// and its row sum to a.work for the merge.
template <int T, bool SPLIT>
__global__ __launch_bounds__(T * 4, 1) void attn_fwd_kernel(AttnArgs a) {
  constexpr int kQW = T / 32;                      // query blocks (waves) of a group
  constexpr int kGroups = 2;                       // key groups
  constexpr int kGThreads = kQW * 64;              // threads of a group
  constexpr int KB = T / 32;                       // 32-key blocks per key tile
  constexpr int kKC = kD / 8;                      // 16-byte chunks per K row
  constexpr int kVC = T / 8;                       // 16-byte chunks per V^T row
  constexpr int kKLoads = T * kKC / kGThreads;     // direct loads per lane for a K tile
  constexpr int kVLoads = kD * kVC / kGThreads;    // and for a V tile
  static_assert(kKLoads == 8 && kVLoads == 8, "load split");
  __shared__ uint4 sK[kGroups][T * kKC];
  __shared__ uint4 sV[kGroups][kD * kVC];
  __shared__ float sML[kQW][2][64];                // group 1's (m, l) for the merge
  static_assert(sizeof(sK) >= size_t(kQW) * 4 * 16 * 64 * 4, "group 1's O fits the K buffers");

  int row = int(blockIdx.x), part = 0;
  bool partial = false;
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
  const int qw = wave % kQW;                       // query block
  const int grp = wave / kQW;                      // key group
  const int lane = tid & 63;
  const int g = lane >> 5;
  const int ln = lane & 31;
  const int qrow = qt * T + qw * 32 + ln;
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
    // Q is in registers before any page copy is issued, so that the only
    // vector-memory operations in flight inside the loop are page copies.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  }

  f32x16 o[kD / 32];
#pragma unroll
  for (int mb = 0; mb < kD / 32; ++mb) o[mb] = f32x16{};
  float m = -INFINITY;   // running (lazily raised) max of raw scores q.k
  float l = 0.f;         // running sum of bf16(exp2((s - m) * c2))

  const int total = ((const const_i32*)a.counts)[row];
  const int first = partial ? int(int64_t(part) * total / a.split) : 0;
  const int count = partial ? int(int64_t(part + 1) * total / a.split) - first : total;
  const const_i32* list = (const const_i32*)a.idx + size_t(row) * a.nk_cap + first;
  const size_t pbytes = page_bytes(T, kD);
  const uint8_t* head_pages = a.pool + (size_t(b) * a.H + h) * a.NT * pbytes;
  const size_t slot_stride = size_t(a.B) * a.H * a.NT * pbytes;
  const float c2 = a.scale_log2;
  const float lazy_raw = kLazyLog2 / fabsf(c2);

  // Entries naming a tile outside the window (stale lists) are skipped: the
  // group idles through that step.
  auto usable = [&](int n) { return n < count && unsigned(list[n]) < unsigned(a.nk); };
  auto page_of = [&](int n) {
    const int j = list[n];
    const int pos = j / a.NT;
    const int t = j - pos * a.NT;
    return head_pages + size_t(a.slot_of[pos]) * slot_stride + size_t(t) * pbytes;
  };
  // Direct HBM -> LDS copies into the group's buffers.  Instruction i of the
  // group's wave w fills the 64 chunks [64*(i*kQW + w), +64) of a buffer; lane
  // l of it fetches the page chunk that the XOR swizzle assigns to that LDS
  // position.  The per-lane byte offsets are loop invariant.
  uint32_t koff[kKLoads], voff[kVLoads];
#pragma unroll
  for (int i = 0; i < kKLoads; ++i) {
    const int p = (i * kQW + qw) * 64 + lane;
    const int r = p / kKC, c = p % kKC;
    koff[i] = uint32_t(r * kKC + (c ^ (r & 15))) * 16u;
  }
#pragma unroll
  for (int i = 0; i < kVLoads; ++i) {
    const int p = (i * kQW + qw) * 64 + lane;
    const int d = p / kVC, c = p % kVC;
    voff[i] = uint32_t(d * kVC + (c ^ (d & (kVC - 1)))) * 16u;
  }
  const uint4* kbuf = sK[grp];
  const uint4* vbuf = sV[grp];
  const uint32_t k_lds = lds_addr(kbuf) + qw * 1024u;
  const uint32_t v_lds = lds_addr(vbuf) + qw * 1024u;
  auto issue_k = [&](const uint8_t* page) {
#pragma unroll
    for (int i = 0; i < kKLoads; ++i) dma16(page, koff[i], k_lds + uint32_t(i * kQW) * 1024u);
  };
  auto issue_v = [&](const uint8_t* page) {
    const uint8_t* vpage = page + size_t(T) * kD * 2;
#pragma unroll
    for (int i = 0; i < kVLoads; ++i) dma16(vpage, voff[i], v_lds + uint32_t(i * kQW) * 1024u);
  };

  // Group grp takes list entries grp, grp + kGroups, ...; both groups run
  // `steps` steps.
  const int steps = (count + kGroups - 1) / kGroups;
  int n = grp;
  bool have = usable(n);
  if (have) {
    const uint8_t* p0 = page_of(n);
    issue_k(p0);
    issue_v(p0);
  }
  for (int step = 0; step < steps; ++step) {
    const int nn = n + kGroups;
    const bool have_next = usable(nn);
    const uint8_t* pnext = have_next ? page_of(nn) : nullptr;
    const int valid = have ? tile_valid(a.tv, list[n] % a.NT, a.NT, a.tail, T) : 0;

    // K_n has landed once only V_n's loads may still be outstanding.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(kVLoads));
    __builtin_amdgcn_s_barrier();

    // S^T = K Q^T : KB blocks of 32 keys x 32 queries.
    f32x16 s[KB];
    if (have) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) s[kb] = f32x16{};
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int ks = 0; ks < kD / 16; ++ks) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const int r = kb * 32 + ln;
          const int cc = 2 * ks + g;
          const bf16x8 kf = as_bf16x8(kbuf[r * kKC + (cc ^ (r & 15))]);
          s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[kb], 0, 0, 0);
        }
      }
      schedule_reads_ahead<KB * kD / 16>();
      __builtin_amdgcn_s_setprio(0);
    }
    // every wave has its K operands in registers: the K buffers can be refilled
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_barrier();
    if (have_next) issue_k(pnext);

    bf16x8 pf[KB][2];
    if (have) {
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
      if (__ballot(mx > m + lazy_raw) != 0) {
        const float mnew = fmaxf(m, mx);
        const float alpha = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((m - mnew) * c2);
        m = mnew;
        l *= alpha;
#pragma unroll
        for (int mb = 0; mb < kD / 32; ++mb) o[mb] *= alpha;
      }
      const float mb2 = m * c2;

      // P^T as the B operand: 16-key halves of each 32-key block.
      float rs = 0.f;
      const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          bf16x2 pr[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][8 * hh + 2 * e], c2, -mb2));
            const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][8 * hh + 2 * e + 1], c2, -mb2));
            pr[e] = bf16x2{(__bf16)p0, (__bf16)p1};
            rs = __builtin_amdgcn_fdot2_f32_bf16(pr[e], ones, rs, false);
          }
          pf[kb][hh] = __builtin_shufflevector(__builtin_shufflevector(pr[0], pr[1], 0, 1, 2, 3),
                                               __builtin_shufflevector(pr[2], pr[3], 0, 1, 2, 3),
                                               0, 1, 2, 3, 4, 5, 6, 7);
        }
      l += pair_sum(rs);
    }

    // V_n has landed once only K_{n+kGroups}'s loads may still be outstanding.
    if (have_next)
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(kKLoads));
    else
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __builtin_amdgcn_s_barrier();

    // O^T += V^T P^T : 4 blocks of 32 dims x 32 queries.
    if (have) {
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int mb = 0; mb < kD / 32; ++mb) {
            const int d = mb * 32 + ln;
            const int cc = 2 * (2 * kb + hh) + g;
            const bf16x8 vf = as_bf16x8(vbuf[d * kVC + (cc ^ (d & (kVC - 1)))]);
            o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kb][hh], o[mb], 0, 0, 0);
          }
      schedule_reads_ahead<KB * 2 * kD / 32>();
      __builtin_amdgcn_s_setprio(0);
    }
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_barrier();
    if (have_next) issue_v(pnext);
    n = nn;
    have = have_next;
  }

  // ---- merge the two key groups: group 1 hands (m, l, O) to group 0 ----
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __syncthreads();   // every copy and operand read of the loop is done
  float* xo = reinterpret_cast<float*>(&sK[0][0]);   // [kQW][4][16][64 lanes]
  if (grp != 0) {
    sML[qw][0][lane] = m;
    sML[qw][1][lane] = l;
#pragma unroll
    for (int mb = 0; mb < kD / 32; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) xo[((qw * 4 + mb) * 16 + e) * 64 + lane] = o[mb][e];
  }
  __syncthreads();
  if (grp != 0) return;
  const float m1 = sML[qw][0][lane], l1 = sML[qw][1][lane];
  const float mm = fmaxf(m, m1);
  const float f0 = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((m - mm) * c2);
  const float f1 = (m1 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((m1 - mm) * c2);
  const float lt = l * f0 + l1 * f1;
  auto merged = [&](int mb, int e) { return o[mb][e] * f0 + xo[((qw * 4 + mb) * 16 + e) * 64 + lane] * f1; };

  if (SPLIT && partial) {
    // partial: O relative to the offset mm*c2 (base 2) and the row sum
    if (qvalid) {
      const size_t wrow = size_t(row - a.split_from) * a.split + part;
      float* op = a.work + (wrow * T + qw * 32 + ln) * kD;
#pragma unroll
      for (int mb = 0; mb < kD / 32; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d0 = mb * 32 + 8 * i + 4 * g;
          *reinterpret_cast<float4*>(op + d0) = make_float4(merged(mb, 4 * i), merged(mb, 4 * i + 1),
                                                            merged(mb, 4 * i + 2), merged(mb, 4 * i + 3));
        }
      if (g == 0) {
        const size_t wrows = (size_t(a.B) * a.H * a.NT - a.split_from) * a.split;
        float2* ml = reinterpret_cast<float2*>(a.work + wrows * T * kD);
        ml[wrow * T + qw * 32 + ln] = make_float2(mm == -INFINITY ? -INFINITY : mm * c2, lt);
      }
    }
    return;
  }
  if (qvalid) {
    const float inv = (lt > 0.f) ? 1.f / lt : 0.f;
    uint16_t* op = a.o + ((size_t(b) * a.L + qrow) * a.H + h) * kD;
#pragma unroll
    for (int mb = 0; mb < kD / 32; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = mb * 32 + 8 * i + 4 * g;
        uint2 u;
        u.x = pack_bf16x2(merged(mb, 4 * i + 0) * inv, merged(mb, 4 * i + 1) * inv);
        u.y = pack_bf16x2(merged(mb, 4 * i + 2) * inv, merged(mb, 4 * i + 3) * inv);
        *reinterpret_cast<uint2*>(op + d0) = u;
      }
    if (a.lse != nullptr && g == 0)
      a.lse[(size_t(b) * a.H + h) * a.L + qrow] = (lt > 0.f) ? mm * a.scale + logf(lt) : -INFINITY;
  }
}

}  // namespace

hipError_t launch_attn_fwd_t64(const AttnArgs& a, hipStream_t stream) {
  const unsigned blocks = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  attn_fwd_kernel<64, false><<<blocks, 256, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_attn_fwd_t64_split(const AttnArgs& a, hipStream_t stream) {
  const unsigned rows = unsigned(a.B) * unsigned(a.H) * unsigned(a.NT);
  const unsigned blocks = unsigned(a.split_from) + (rows - unsigned(a.split_from)) * unsigned(a.split);
  attn_fwd_kernel<64, true><<<blocks, 256, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_attn_split_merge(a, stream);
}

}  // namespace uf
