// C ABI of the block-sparse chunk-causal attention path: argument validation,
// the window (ring) metadata, and kernel launches.  See include/uf.h for the
// contract of every entry point.
//
// The window realises the paper's compact KV cache window of the SR model
// (Sec. 2.3.2, dynamic cache management (iii); App. C) as a
// fixed set of slots in a caller-owned pool: each live chunk occupies one slot;
// logical order is ascending append sequence number, so an optional pinned
// first chunk always sits at logical position 0; eviction frees the oldest
// non-pinned slots and moves no data.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "launch.h"
#include "launch_bwd.h"

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int ok() {
  g_last_error[0] = '\0';
  return UF_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct Live {
  int32_t slot;
  int64_t seq;
  bool sink;
};

int check_desc(const uf_kv_desc* d) {
  if (d == nullptr) return fail(UF_ERR_ARG, "desc is null");
  if (d->batch < 1) return fail(UF_ERR_ARG, "batch must be >= 1 (got %d)", d->batch);
  if (d->heads < 1) return fail(UF_ERR_ARG, "heads must be >= 1 (got %d)", d->heads);
  if (d->chunk_tokens < 1) return fail(UF_ERR_ARG, "chunk_tokens must be >= 1 (got %d)", d->chunk_tokens);
  if (d->max_chunks < 1 || d->max_chunks > UF_MAX_CHUNKS)
    return fail(UF_ERR_ARG, "max_chunks must be in [1, %d] (got %d)", UF_MAX_CHUNKS, d->max_chunks);
  if (d->pin_sink != 0 && d->pin_sink != 1) return fail(UF_ERR_ARG, "pin_sink must be 0 or 1");
  if (d->flags & ~(UF_F_DRYRUN | UF_F_POISON_PAD)) return fail(UF_ERR_ARG, "unknown flag bits 0x%x", d->flags);
  if (d->head_dim != 128) return fail(UF_ERR_UNSUPPORTED, "head_dim must be 128 (got %d)", d->head_dim);
  if (d->tile != 64 && d->tile != 128) return fail(UF_ERR_UNSUPPORTED, "tile must be 64 or 128 (got %d)", d->tile);
  // Index arithmetic in the kernels: element offsets are 64-bit, but list
  // rows, page counts and token indices must fit in 31 bits.
  const int64_t nt = (int64_t(d->chunk_tokens) + d->tile - 1) / d->tile;
  const int64_t rows = int64_t(d->batch) * d->heads * nt;
  const int64_t tokens = int64_t(d->batch) * d->chunk_tokens;
  if (rows * d->max_chunks > INT32_MAX || tokens * d->heads > INT32_MAX)
    return fail(UF_ERR_ARG, "shape too large: B*H*NT*max_chunks and B*L*H must fit in int32");
  return UF_OK;
}

}  // namespace

struct uf_kv {
  uf_kv_desc d;
  uint8_t* pool;
  // block geometry (uf_kv_set_block_geom): tiles are 3-D blocks
  bool blocked = false;
  uf_block_geom geom{};
  int32_t nbh = 0, nbw = 0;
  uint8_t block_valid[UF_MAX_BLOCKS] = {};
  uf::TileValid tile_valid(int32_t local_r) const {
    uf::TileValid v{};
    v.blocked = blocked ? 1 : 0;
    v.nbh = blocked ? nbh : 1;
    v.nbw = blocked ? nbw : 1;
    v.local_half = (blocked && local_r > 0) ? local_r / 2 : -1;
    if (blocked)
      for (int32_t j = 0; j < UF_MAX_BLOCKS; ++j) v.count4[j >> 2] |= uint32_t(block_valid[j]) << (8 * (j & 3));
    return v;
  }
  // pooled keys follow the pages: [max_chunks][B][H][NT][D] float32
  float* kmean() const {
    const size_t pages = size_t(d.max_chunks) * d.batch * d.heads * nt;
    return reinterpret_cast<float*>(pool + pages * uf::page_bytes(d.tile, d.head_dim));
  }
  size_t pool_bytes;
  int32_t nt;
  int32_t tail;
  int32_t nk_cap;
  int32_t mask_words;
  std::vector<Live> live;       // logical order
  std::vector<uint8_t> used;    // per slot
  int64_t next_seq;

  bool dry() const { return (d.flags & UF_F_DRYRUN) != 0; }
  int32_t rows() const { return d.batch * d.heads * nt; }
  uf_lists_layout layout() const {
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    uf_lists_layout lay{};
    lay.rows = rows();
    lay.nk_cap = nk_cap;
    lay.mask_words = mask_words;
    lay.counts_offset = 0;
    lay.idx_offset = up(size_t(lay.rows) * 4);
    lay.mask_offset = lay.idx_offset + up(size_t(lay.rows) * size_t(nk_cap) * 4);
    lay.scratch_offset = lay.mask_offset + up(size_t(lay.rows) * size_t(mask_words) * 4);
    lay.total_bytes = lay.scratch_offset + up(size_t(lay.rows) * size_t(d.head_dim) * 4);
    return lay;
  }
};

namespace {

int check_geom(const uf_block_geom* g, int32_t* padded, int32_t* nblocks) {
  if (g == nullptr) return fail(UF_ERR_ARG, "geometry is null");
  if (g->frames < 1 || g->grid_h < 1 || g->grid_w < 1 || g->bt < 1 || g->bh < 1 || g->bw < 1)
    return fail(UF_ERR_ARG, "geometry fields must be >= 1");
  const int64_t nb = int64_t((g->frames + g->bt - 1) / g->bt) * ((g->grid_h + g->bh - 1) / g->bh) *
                     ((g->grid_w + g->bw - 1) / g->bw);
  const int64_t tile = int64_t(g->bt) * g->bh * g->bw;
  if (nb > UF_MAX_BLOCKS) return fail(UF_ERR_UNSUPPORTED, "%lld blocks per chunk, at most %d", (long long)nb, UF_MAX_BLOCKS);
  if (tile > 255) return fail(UF_ERR_UNSUPPORTED, "blocks of %lld tokens, at most 255", (long long)tile);
  if (nb * tile > INT32_MAX) return fail(UF_ERR_ARG, "block-order length too large");
  if (padded) *padded = int32_t(nb * tile);
  if (nblocks) *nblocks = int32_t(nb);
  return UF_OK;
}

int check_local(const uf_kv* kv, int32_t local_r) {
  if (local_r == 0) return UF_OK;
  if (local_r < 0 || local_r % 2 == 0) return fail(UF_ERR_ARG, "local_r must be 0 or odd and positive (got %d)", local_r);
  if (!kv->blocked) return fail(UF_ERR_ARG, "local_r needs block geometry (uf_kv_set_block_geom)");
  return UF_OK;
}

}  // namespace

extern "C" {

int uf_kv_pool_bytes(const uf_kv_desc* desc, size_t* bytes) {
  if (int s = check_desc(desc)) return s;
  if (bytes == nullptr) return fail(UF_ERR_ARG, "bytes is null");
  const size_t nt = (size_t(desc->chunk_tokens) + desc->tile - 1) / desc->tile;
  const size_t pages = size_t(desc->max_chunks) * desc->batch * desc->heads * nt;
  *bytes = pages * (uf::page_bytes(desc->tile, desc->head_dim) + size_t(4) * desc->head_dim);
  return ok();
}

int uf_kv_create(const uf_kv_desc* desc, void* d_pool, size_t pool_bytes, uf_kv** out) {
  if (out == nullptr) return fail(UF_ERR_ARG, "out is null");
  size_t need = 0;
  if (int s = uf_kv_pool_bytes(desc, &need)) return s;
  const bool dry = (desc->flags & UF_F_DRYRUN) != 0;
  if (!dry && d_pool == nullptr) return fail(UF_ERR_ARG, "pool is null");
  if (d_pool != nullptr && !aligned(d_pool, 256)) return fail(UF_ERR_ARG, "pool must be 256-byte aligned");
  if (!dry && pool_bytes < need)
    return fail(UF_ERR_CAPACITY, "pool has %zu bytes, window needs %zu", pool_bytes, need);
  uf_kv* kv = new (std::nothrow) uf_kv();
  if (kv == nullptr) return fail(UF_ERR_ARG, "out of host memory");
  kv->d = *desc;
  kv->pool = static_cast<uint8_t*>(d_pool);
  kv->pool_bytes = pool_bytes;
  kv->nt = (desc->chunk_tokens + desc->tile - 1) / desc->tile;
  kv->tail = desc->chunk_tokens - (kv->nt - 1) * desc->tile;
  kv->nk_cap = desc->max_chunks * kv->nt;
  kv->mask_words = (kv->nk_cap + 31) / 32;
  kv->used.assign(size_t(desc->max_chunks), 0);
  kv->next_seq = 0;
  *out = kv;
  return ok();
}

int uf_kv_destroy(uf_kv* kv) {
  delete kv;
  return ok();
}

namespace {

// Copy one chunk's K and V into the pages (and pooled keys) of `slot`.
int write_chunk(uf_kv* kv, int32_t slot, const void* d_k, const void* d_v, void* stream) {
  if (!kv->dry()) {
    if (d_k == nullptr || d_v == nullptr) return fail(UF_ERR_ARG, "k or v is null");
    if (!aligned(d_k, 16) || !aligned(d_v, 16)) return fail(UF_ERR_ARG, "k and v must be 16-byte aligned");
    uf::AppendArgs a{};
    a.k = static_cast<const uint16_t*>(d_k);
    a.v = static_cast<const uint16_t*>(d_v);
    a.pool = kv->pool;
    a.kmean = kv->kmean();
    a.slot = slot;
    a.B = kv->d.batch;
    a.H = kv->d.heads;
    a.L = kv->d.chunk_tokens;
    a.T = kv->d.tile;
    a.NT = kv->nt;
    a.tail = kv->tail;
    a.pad = (kv->d.flags & UF_F_POISON_PAD) ? uint16_t(0x461C) : uint16_t(0);  // bf16 9984.0
    a.tv = kv->tile_valid(0);
    hipError_t e = uf::launch_kv_append(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(UF_ERR_HIP, "kv_append launch: %s", hipGetErrorString(e));
  }
  return UF_OK;
}

}  // namespace

int uf_kv_append(uf_kv* kv, const void* d_k, const void* d_v, void* stream) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  if (int32_t(kv->live.size()) >= kv->d.max_chunks)
    return fail(UF_ERR_CAPACITY, "window full (%d chunks)", kv->d.max_chunks);
  int32_t slot = 0;
  while (kv->used[size_t(slot)]) ++slot;
  if (int s = write_chunk(kv, slot, d_k, d_v, stream)) return s;
  const int64_t seq = kv->next_seq++;
  kv->used[size_t(slot)] = 1;
  kv->live.push_back(Live{slot, seq, kv->d.pin_sink == 1 && seq == 0});
  return ok();
}

int uf_kv_replace_newest(uf_kv* kv, const void* d_k, const void* d_v, void* stream) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  if (kv->live.empty()) return fail(UF_ERR_EMPTY, "window holds no chunk");
  if (int s = write_chunk(kv, kv->live.back().slot, d_k, d_v, stream)) return s;
  return ok();
}

int uf_kv_evict(uf_kv* kv, int32_t n_chunks) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  if (n_chunks < 0) return fail(UF_ERR_ARG, "n_chunks must be >= 0 (got %d)", n_chunks);
  int32_t evictable = 0;
  for (const Live& c : kv->live) evictable += c.sink ? 0 : 1;
  if (n_chunks > evictable)
    return fail(UF_ERR_EMPTY, "asked to evict %d chunks, %d evictable", n_chunks, evictable);
  std::vector<Live> keep;
  keep.reserve(kv->live.size());
  int32_t dropped = 0;
  for (const Live& c : kv->live) {
    if (!c.sink && dropped < n_chunks) {
      kv->used[size_t(c.slot)] = 0;
      ++dropped;
    } else {
      keep.push_back(c);
    }
  }
  kv->live.swap(keep);
  return ok();
}

int uf_kv_get_info(const uf_kv* kv, uf_kv_info* info) {
  if (kv == nullptr || info == nullptr) return fail(UF_ERR_ARG, "null argument");
  info->n_live = int32_t(kv->live.size());
  info->nq_tiles = kv->nt;
  info->nk_tiles = info->n_live * kv->nt;
  info->tail_valid = kv->tail;
  info->first_seq = kv->live.empty() ? -1 : kv->live.front().seq;
  info->last_seq = kv->live.empty() ? -1 : kv->live.back().seq;
  info->has_sink = (!kv->live.empty() && kv->live.front().sink) ? 1 : 0;
  info->nk_cap = kv->nk_cap;
  return ok();
}

int uf_kv_logical(const uf_kv* kv, int32_t pos, int32_t* slot, int64_t* seq) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  if (pos < 0 || pos >= int32_t(kv->live.size()))
    return fail(UF_ERR_ARG, "logical position %d outside [0, %zu)", pos, kv->live.size());
  if (slot) *slot = kv->live[size_t(pos)].slot;
  if (seq) *seq = kv->live[size_t(pos)].seq;
  return ok();
}

int uf_tile_lists_layout(const uf_kv* kv, uf_lists_layout* layout) {
  if (kv == nullptr || layout == nullptr) return fail(UF_ERR_ARG, "null argument");
  *layout = kv->layout();
  return ok();
}

int uf_tile_lists_bytes(const uf_kv* kv, size_t* bytes) {
  if (kv == nullptr || bytes == nullptr) return fail(UF_ERR_ARG, "null argument");
  *bytes = kv->layout().total_bytes;
  return ok();
}

int uf_build_tile_lists(const uf_kv* kv, const uf_keep_rule* rule, void* d_lists, size_t bytes,
                        void* stream) {
  if (kv == nullptr || rule == nullptr) return fail(UF_ERR_ARG, "null argument");
  if (!(rule->p_prior >= 0.0 && rule->p_prior <= 1.0))
    return fail(UF_ERR_ARG, "p_prior must lie in [0, 1]");
  if ((rule->keep_sink != 0 && rule->keep_sink != 1) || (rule->keep_current != 0 && rule->keep_current != 1))
    return fail(UF_ERR_ARG, "keep_sink and keep_current must be 0 or 1");
  if (rule->reserved != 0) return fail(UF_ERR_ARG, "reserved must be 0");
  if (int s = check_local(kv, rule->local_r)) return s;
  if (kv->live.empty()) return fail(UF_ERR_EMPTY, "window holds no chunk");
  const uf_lists_layout lay = kv->layout();
  if (kv->dry()) return ok();
  if (d_lists == nullptr || !aligned(d_lists, 256)) return fail(UF_ERR_ARG, "lists must be non-null and 256-byte aligned");
  if (bytes < lay.total_bytes) return fail(UF_ERR_ARG, "lists buffer has %zu bytes, needs %zu", bytes, lay.total_bytes);
  uf::ListArgs a{};
  a.tv = kv->tile_valid(rule->local_r);
  a.lists = static_cast<uint8_t*>(d_lists);
  a.idx_offset = lay.idx_offset;
  a.mask_offset = lay.mask_offset;
  a.rows = lay.rows;
  a.H = kv->d.heads;
  a.NT = kv->nt;
  a.nk = int32_t(kv->live.size()) * kv->nt;
  a.nk_cap = kv->nk_cap;
  a.mask_words = kv->mask_words;
  a.seed = rule->seed;
  a.thr = (rule->p_prior >= 1.0) ? (uint64_t(1) << 32) : uint64_t(std::floor(rule->p_prior * 4294967296.0));
  a.keep_sink = rule->keep_sink;
  a.keep_current = rule->keep_current;
  a.cur_seq = kv->live.back().seq;
  for (size_t p = 0; p < kv->live.size(); ++p) {
    a.seq[p] = kv->live[p].seq;
    a.sink[p] = kv->live[p].sink ? 1 : 0;
  }
  hipError_t e = uf::launch_tile_lists(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(UF_ERR_HIP, "tile_lists launch: %s", hipGetErrorString(e));
  return ok();
}

int uf_build_topk_lists(const uf_kv* kv, const void* d_q, const uf_topk_rule* rule, void* d_lists,
                        size_t bytes, void* stream) {
  if (kv == nullptr || rule == nullptr) return fail(UF_ERR_ARG, "null argument");
  if (rule->budget < 0) return fail(UF_ERR_ARG, "budget must be >= 0 (got %d)", rule->budget);
  if ((rule->keep_sink != 0 && rule->keep_sink != 1) || (rule->keep_current != 0 && rule->keep_current != 1))
    return fail(UF_ERR_ARG, "keep_sink and keep_current must be 0 or 1");
  if (int s = check_local(kv, rule->local_r)) return s;
  if (kv->live.empty()) return fail(UF_ERR_EMPTY, "window holds no chunk");
  const int32_t nk = int32_t(kv->live.size()) * kv->nt;
  const int32_t lo = (kv->live.front().sink && rule->keep_sink) ? kv->nt : 0;
  const int32_t hi = rule->keep_current ? nk - kv->nt : nk;
  const int32_t nc = std::max(hi - lo, 0);
  if (nc > uf::kTopkMaxCandidates)
    return fail(UF_ERR_UNSUPPORTED, "%d ranked candidates per row, at most %d", nc, uf::kTopkMaxCandidates);
  const uf_lists_layout lay = kv->layout();
  if (kv->dry()) return ok();
  if (d_q == nullptr || !aligned(d_q, 16)) return fail(UF_ERR_ARG, "q must be non-null and 16-byte aligned");
  if (d_lists == nullptr || !aligned(d_lists, 256)) return fail(UF_ERR_ARG, "lists must be non-null and 256-byte aligned");
  if (bytes < lay.total_bytes) return fail(UF_ERR_ARG, "lists buffer has %zu bytes, needs %zu", bytes, lay.total_bytes);
  uf::TopkArgs a{};
  a.q = static_cast<const uint16_t*>(d_q);
  a.kmean = kv->kmean();
  a.lists = static_cast<uint8_t*>(d_lists);
  a.idx_offset = lay.idx_offset;
  a.mask_offset = lay.mask_offset;
  a.scratch_offset = lay.scratch_offset;
  a.B = kv->d.batch;
  a.H = kv->d.heads;
  a.L = kv->d.chunk_tokens;
  a.T = kv->d.tile;
  a.NT = kv->nt;
  a.tail = kv->tail;
  a.nk = nk;
  a.nk_cap = kv->nk_cap;
  a.mask_words = kv->mask_words;
  a.G = std::max(1, std::min({2, kv->nt, uf::kTopkMaxCandidates / std::max(nc, 1)}));
  a.cand_lo = lo;
  a.cand_hi = hi;
  a.budget = rule->budget;
  a.tv = kv->tile_valid(rule->local_r);
  for (size_t p = 0; p < kv->live.size(); ++p) a.slot_of[p] = kv->live[p].slot;
  const size_t lds = std::max<size_t>(size_t(a.G) * size_t(nc) * 5, 16);
  hipError_t e = uf::launch_topk_lists(a, lds, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(UF_ERR_HIP, "topk_lists launch: %s", hipGetErrorString(e));
  return ok();
}

int uf_topk_budget(double rho, int64_t seq_len, int64_t seq_ref, int64_t n_blocks, int32_t k_min,
                   int32_t* budget) {
  if (budget == nullptr) return fail(UF_ERR_ARG, "budget is null");
  if (!(std::isfinite(rho) && rho >= 0.0)) return fail(UF_ERR_ARG, "rho must be finite and >= 0");
  if (seq_ref < 1 || seq_len < 0 || n_blocks < 0 || k_min < 0)
    return fail(UF_ERR_ARG, "seq_ref must be >= 1 and the counts >= 0");
  const double k = std::floor(rho * double(seq_len) / double(seq_ref) * double(n_blocks));
  const double c = std::min(std::max(k, double(k_min)), double(INT32_MAX));
  *budget = int32_t(c);
  return ok();
}

namespace {

// Validation and arguments shared by the attention entry points.
int attn_args(const uf_kv* kv, const void* d_q, const void* d_lists, float scale, void* d_o, float* d_lse,
              uf::AttnArgs* out) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  if (!(std::isfinite(scale) && scale > 0.f && std::isnormal(scale * 1.4426950408889634f)))
    return fail(UF_ERR_ARG, "scale must be positive, finite and normal");
  if (kv->live.empty()) return fail(UF_ERR_EMPTY, "window holds no chunk");
  if (kv->dry()) return UF_OK;
  if (d_q == nullptr || d_o == nullptr || d_lists == nullptr) return fail(UF_ERR_ARG, "q, o or lists is null");
  if (!aligned(d_q, 16) || !aligned(d_o, 16)) return fail(UF_ERR_ARG, "q and o must be 16-byte aligned");
  if (!aligned(d_lists, 256)) return fail(UF_ERR_ARG, "lists must be 256-byte aligned");
  if (d_lse != nullptr && !aligned(d_lse, 4)) return fail(UF_ERR_ARG, "lse must be 4-byte aligned");
  const uf_lists_layout lay = kv->layout();
  uf::AttnArgs a{};
  a.q = static_cast<const uint16_t*>(d_q);
  a.o = static_cast<uint16_t*>(d_o);
  a.lse = d_lse;
  a.pool = kv->pool;
  a.counts = reinterpret_cast<const int32_t*>(static_cast<const uint8_t*>(d_lists) + lay.counts_offset);
  a.idx = reinterpret_cast<const int32_t*>(static_cast<const uint8_t*>(d_lists) + lay.idx_offset);
  a.B = kv->d.batch;
  a.H = kv->d.heads;
  a.L = kv->d.chunk_tokens;
  a.T = kv->d.tile;
  a.NT = kv->nt;
  a.nt_div = UINT64_MAX / uint64_t(kv->nt);
  a.tail = kv->tail;
  a.nk = int32_t(kv->live.size()) * kv->nt;
  a.nk_cap = kv->nk_cap;
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.split = 1;
  a.split_from = 0;
  a.work = nullptr;
  a.tv = kv->tile_valid(0);
  for (size_t p = 0; p < kv->live.size(); ++p) a.slot_of[p] = kv->live[p].slot;
  *out = a;
  return UF_OK;
}

// Partials of the rows split_from .. rows-1, n_split slices each.
size_t split_work_bytes(const uf_kv* kv, int32_t n_split, int32_t split_from = 0) {
  const size_t rows = size_t(kv->layout().rows) - size_t(split_from);
  return rows * size_t(n_split) * size_t(kv->d.tile) * (size_t(kv->d.head_dim) + 2) * 4;
}

}  // namespace

int uf_sparse_causal_attn_fwd(const uf_kv* kv, const void* d_q, const void* d_lists, float scale,
                              void* d_o, float* d_lse, void* stream) {
  uf::AttnArgs a{};
  if (int s = attn_args(kv, d_q, d_lists, scale, d_o, d_lse, &a)) return s;
  if (kv->dry()) return ok();
  hipError_t e = uf::launch_attn_fwd(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(UF_ERR_HIP, "attn_fwd launch: %s", hipGetErrorString(e));
  return ok();
}

int uf_attn_split_work_bytes(const uf_kv* kv, int32_t n_split, size_t* bytes) {
  if (kv == nullptr || bytes == nullptr) return fail(UF_ERR_ARG, "null argument");
  if (n_split < 1 || n_split > UF_MAX_SPLIT) return fail(UF_ERR_ARG, "n_split must be in [1, %d]", UF_MAX_SPLIT);
  *bytes = split_work_bytes(kv, n_split);
  return ok();
}

int uf_sparse_causal_attn_fwd_split(const uf_kv* kv, const void* d_q, const void* d_lists, float scale,
                                    void* d_o, float* d_lse, int32_t n_split, void* d_work, size_t work_bytes,
                                    void* stream) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  if (n_split < 1 || n_split > UF_MAX_SPLIT) return fail(UF_ERR_ARG, "n_split must be in [1, %d]", UF_MAX_SPLIT);
  uf::AttnArgs a{};
  if (int s = attn_args(kv, d_q, d_lists, scale, d_o, d_lse, &a)) return s;
  if (kv->dry()) return ok();
  if (d_work == nullptr || !aligned(d_work, 16)) return fail(UF_ERR_ARG, "work must be non-null and 16-byte aligned");
  if (work_bytes < split_work_bytes(kv, n_split))
    return fail(UF_ERR_ARG, "work has %zu bytes, needs %zu", work_bytes, split_work_bytes(kv, n_split));
  a.split = n_split;
  a.work = static_cast<float*>(d_work);
  hipError_t e = uf::launch_attn_fwd_split(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(UF_ERR_HIP, "attn_fwd split launch: %s", hipGetErrorString(e));
  return ok();
}

int uf_attn_tail_plan(const uf_kv* kv, int32_t n_cu, int32_t* split_from, int32_t* n_split) {
  if (kv == nullptr || split_from == nullptr || n_split == nullptr) return fail(UF_ERR_ARG, "null argument");
  if (n_cu < 1) return fail(UF_ERR_ARG, "n_cu must be >= 1");
  // workgroups resident at once: one per CU with either tile size
  const int64_t R = kv->layout().rows, C = int64_t(n_cu);
  *split_from = int32_t(R);
  *n_split = 1;
  // time in row-times with rounds of C workgroups: whole rows take
  // ceil(R / C); rows F.. cut into S slices take F / C + ceil((R - F) * S / C)
  // rounds of 1/S row-time plus a slice's fixed cost, and the merge launch
  // follows (F = C * floor(R / C)).  The fixed costs, in key tiles of work
  // (a row of the window is taken as dense, nk tiles), are measured ones: a
  // slice's prologue and epilogue about 9 tiles, the merge about 12.
  constexpr double kSliceTiles = 9.0, kMergeTiles = 12.0;
  const int64_t q = R / C, r = R % C;
  if (r == 0) return ok();
  const double whole = double(q + 1);
  // no more slices than key tiles in the window, so that no slice is empty by construction
  const int64_t nk = int64_t(kv->live.size()) * kv->nt;
  const int64_t s_max = std::min<int64_t>(nk, q == 0 ? std::min<int64_t>(UF_MAX_SPLIT, std::max<int64_t>(2, C / R)) : 8);
  double best = whole;
  int32_t best_s = 1;
  for (int64_t S = 2; S <= s_max; ++S) {
    const double cost = double(q) + double((r * S + C - 1) / C) * (1.0 / double(S) + kSliceTiles / double(nk)) +
                        kMergeTiles / double(nk);
    if (cost < best - 1e-9) {
      best = cost;
      best_s = int32_t(S);
    }
  }
  // not worth the merge launch and the slices' fixed costs: under a fifth of
  // a row-time, or under 16 key tiles of one row's work, saved
  if (best > whole - 0.2 || (whole - best) * double(nk) < 16.0) return ok();
  *split_from = int32_t(q * C);
  *n_split = best_s;
  return ok();
}

int uf_attn_split_rows_work_bytes(const uf_kv* kv, int32_t split_from, int32_t n_split, size_t* bytes) {
  if (kv == nullptr || bytes == nullptr) return fail(UF_ERR_ARG, "null argument");
  if (n_split < 1 || n_split > UF_MAX_SPLIT) return fail(UF_ERR_ARG, "n_split must be in [1, %d]", UF_MAX_SPLIT);
  if (split_from < 0 || split_from > kv->layout().rows)
    return fail(UF_ERR_ARG, "split_from must be in [0, %d]", kv->layout().rows);
  *bytes = split_work_bytes(kv, n_split, split_from);
  return ok();
}

int uf_sparse_causal_attn_fwd_split_rows(const uf_kv* kv, const void* d_q, const void* d_lists, float scale,
                                         void* d_o, float* d_lse, int32_t split_from, int32_t n_split,
                                         void* d_work, size_t work_bytes, void* stream) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  if (n_split < 1 || n_split > UF_MAX_SPLIT) return fail(UF_ERR_ARG, "n_split must be in [1, %d]", UF_MAX_SPLIT);
  if (split_from < 0 || split_from > kv->layout().rows)
    return fail(UF_ERR_ARG, "split_from must be in [0, %d]", kv->layout().rows);
  uf::AttnArgs a{};
  if (int s = attn_args(kv, d_q, d_lists, scale, d_o, d_lse, &a)) return s;
  if (kv->dry()) return ok();
  const size_t need = split_work_bytes(kv, n_split, split_from);
  if (need > 0 && (d_work == nullptr || !aligned(d_work, 16)))
    return fail(UF_ERR_ARG, "work must be non-null and 16-byte aligned");
  if (work_bytes < need) return fail(UF_ERR_ARG, "work has %zu bytes, needs %zu", work_bytes, need);
  a.split = n_split;
  a.split_from = split_from;
  a.work = static_cast<float*>(d_work);
  hipError_t e = uf::launch_attn_fwd_split(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(UF_ERR_HIP, "attn_fwd split launch: %s", hipGetErrorString(e));
  return ok();
}

namespace {

// One query-tile record per list row.
size_t bwd_work_bytes(const uf_kv* kv) { return size_t(kv->layout().rows) * uf::kBwdQTile; }

}  // namespace

int uf_attn_bwd_work_bytes(const uf_kv* kv, size_t* bytes) {
  if (kv == nullptr || bytes == nullptr) return fail(UF_ERR_ARG, "null argument");
  *bytes = bwd_work_bytes(kv);
  return ok();
}

namespace {

// Validation and kernel arguments shared by both backward entry points; the
// caller's workspace is checked (and set) only when `work` is true.
int bwd_args(const uf_kv* kv, const void* d_q, const void* d_o, const void* d_do, const float* d_lse,
             const void* d_lists, float scale, float* d_dq, float* d_dk, float* d_dv, bool work, void* d_work,
             size_t work_bytes, uf::BwdArgs* out) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  if (kv->nt > uf::kBwdMaxQTiles) return fail(UF_ERR_UNSUPPORTED, "the backward handles at most %d query tiles", uf::kBwdMaxQTiles);
  uf::AttnArgs f{};
  if (int s = attn_args(kv, d_q, d_lists, scale, const_cast<void*>(d_o), const_cast<float*>(d_lse), &f)) return s;
  if (kv->dry()) return ok();
  if (d_do == nullptr || d_lse == nullptr || d_dq == nullptr || d_dk == nullptr || d_dv == nullptr)
    return fail(UF_ERR_ARG, "do, lse, dq, dk or dv is null");
  if (!aligned(d_do, 16) || !aligned(d_dq, 16) || !aligned(d_dk, 16) || !aligned(d_dv, 16))
    return fail(UF_ERR_ARG, "do, dq, dk and dv must be 16-byte aligned");
  if (work) {
    if (d_work == nullptr || !aligned(d_work, 16)) return fail(UF_ERR_ARG, "work must be non-null and 16-byte aligned");
    if (work_bytes < bwd_work_bytes(kv))
      return fail(UF_ERR_ARG, "work has %zu bytes, needs %zu", work_bytes, bwd_work_bytes(kv));
  }
  const uf_lists_layout lay = kv->layout();
  if (int64_t(lay.rows) * int64_t(kv->live.size()) > INT32_MAX) return fail(UF_ERR_ARG, "shape too large");
  uf::BwdArgs& a = *out;
  a.q = f.q;
  a.o = f.o;
  a.dout = static_cast<const uint16_t*>(d_do);
  a.lse = d_lse;
  a.pool = kv->pool;
  a.counts = f.counts;
  a.idx = f.idx;
  a.mask = reinterpret_cast<const uint32_t*>(static_cast<const uint8_t*>(d_lists) + lay.mask_offset);
  a.dq = d_dq;
  a.dk = d_dk;
  a.dv = d_dv;
  a.work = static_cast<uint8_t*>(d_work);
  a.B = f.B;
  a.H = f.H;
  a.L = f.L;
  a.T = f.T;
  a.NT = f.NT;
  a.tail = f.tail;
  a.nk = f.nk;
  a.nk_cap = f.nk_cap;
  a.mask_words = int32_t(lay.mask_words);
  a.n_live = int32_t(kv->live.size());
  a.scale = f.scale;
  a.scale_log2 = f.scale_log2;
  for (int p = 0; p < a.n_live; ++p) a.slot_of[p] = f.slot_of[p];
  a.tv = f.tv;
  return ok();
}

}  // namespace

int uf_sparse_causal_attn_bwd(const uf_kv* kv, const void* d_q, const void* d_o, const void* d_do,
                              const float* d_lse, const void* d_lists, float scale, float* d_dq, float* d_dk,
                              float* d_dv, void* d_work, size_t work_bytes, void* stream) {
  uf::BwdArgs a{};
  if (int s = bwd_args(kv, d_q, d_o, d_do, d_lse, d_lists, scale, d_dq, d_dk, d_dv, true, d_work, work_bytes, &a))
    return s;
  if (kv->dry()) return ok();
  hipError_t e = uf::launch_attn_bwd(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(UF_ERR_HIP, "attn_bwd launch: %s", hipGetErrorString(e));
  return ok();
}

int uf_sparse_causal_attn_bwd_noalloc(const uf_kv* kv, const void* d_q, const void* d_o, const void* d_do,
                                      const float* d_lse, const void* d_lists, float scale, float* d_dq,
                                      float* d_dk, float* d_dv, void* stream) {
  if (kv != nullptr && kv->d.tile == 128 && bwd_work_bytes(kv) > uf::kBwdScratchBytes)
    return fail(UF_ERR_CAPACITY, "the backward of %d list rows needs %zu bytes of scratch, the library holds %zu "
                "(at most %zu rows)", kv->layout().rows, bwd_work_bytes(kv), uf::kBwdScratchBytes,
                uf::kBwdScratchBytes / uf::kBwdQTile);
  uf::BwdArgs a{};
  if (int s = bwd_args(kv, d_q, d_o, d_do, d_lse, d_lists, scale, d_dq, d_dk, d_dv, false, nullptr, 0, &a))
    return s;
  if (kv->dry()) return ok();
  hipError_t e = uf::launch_attn_bwd_noalloc(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(UF_ERR_HIP, "attn_bwd (no-allocation) launch: %s", hipGetErrorString(e));
  return ok();
}

int uf_block_geom_tokens(const uf_block_geom* g, int32_t* padded_tokens, int32_t* n_blocks) {
  if (int s = check_geom(g, padded_tokens, n_blocks)) return s;
  return ok();
}

int uf_kv_set_block_geom(uf_kv* kv, const uf_block_geom* g) {
  if (kv == nullptr) return fail(UF_ERR_ARG, "handle is null");
  int32_t padded = 0, nb = 0;
  if (int s = check_geom(g, &padded, &nb)) return s;
  if (!kv->live.empty() || kv->next_seq != 0) return fail(UF_ERR_ARG, "block geometry must be set on a new, empty window");
  if (g->bt * g->bh * g->bw != kv->d.tile)
    return fail(UF_ERR_ARG, "block of %d tokens, tile is %d", g->bt * g->bh * g->bw, kv->d.tile);
  if (padded != kv->d.chunk_tokens)
    return fail(UF_ERR_ARG, "chunk_tokens must be the block-order length %d (got %d)", padded, kv->d.chunk_tokens);
  kv->blocked = true;
  kv->geom = *g;
  kv->nbh = (g->grid_h + g->bh - 1) / g->bh;
  kv->nbw = (g->grid_w + g->bw - 1) / g->bw;
  for (int32_t j = 0; j < nb; ++j) {
    const int32_t bti = j / (kv->nbh * kv->nbw), bhi = (j / kv->nbw) % kv->nbh, bwi = j % kv->nbw;
    const int32_t n = std::min(g->bt, g->frames - bti * g->bt) * std::min(g->bh, g->grid_h - bhi * g->bh) *
                      std::min(g->bw, g->grid_w - bwi * g->bw);
    kv->block_valid[j] = uint8_t(n);
  }
  return ok();
}

int uf_block_permute(const uf_block_geom* g, int32_t batch, int32_t heads, int32_t head_dim, const void* d_src,
                     void* d_dst, int32_t inverse, void* stream) {
  int32_t padded = 0, nb = 0;
  if (int s = check_geom(g, &padded, &nb)) return s;
  if (batch < 1 || heads < 1) return fail(UF_ERR_ARG, "batch and heads must be >= 1");
  if (head_dim != 128) return fail(UF_ERR_UNSUPPORTED, "head_dim must be 128 (got %d)", head_dim);
  if (inverse != 0 && inverse != 1) return fail(UF_ERR_ARG, "inverse must be 0 or 1");
  const int64_t tokens = int64_t(g->frames) * g->grid_h * g->grid_w;
  if (int64_t(batch) * padded * heads > INT32_MAX) return fail(UF_ERR_ARG, "shape too large");
  if (d_src == nullptr || d_dst == nullptr || !aligned(d_src, 16) || !aligned(d_dst, 16))
    return fail(UF_ERR_ARG, "src and dst must be non-null and 16-byte aligned");
  uf::PermuteArgs a{};
  a.src = static_cast<const uint16_t*>(d_src);
  a.dst = static_cast<uint16_t*>(d_dst);
  a.B = batch;
  a.H = heads;
  a.frames = g->frames;
  a.gh = g->grid_h;
  a.gw = g->grid_w;
  a.bt = g->bt;
  a.bh = g->bh;
  a.bw = g->bw;
  a.nbh = (g->grid_h + g->bh - 1) / g->bh;
  a.nbw = (g->grid_w + g->bw - 1) / g->bw;
  a.tokens = int32_t(tokens);
  a.padded = padded;
  a.inverse = inverse;
  hipError_t e = uf::launch_block_permute(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(UF_ERR_HIP, "block_permute launch: %s", hipGetErrorString(e));
  return ok();
}

const char* uf_status_string(int status) {
  switch (status) {
    case UF_OK: return "UF_OK";
    case UF_ERR_ARG: return "UF_ERR_ARG: invalid argument";
    case UF_ERR_UNSUPPORTED: return "UF_ERR_UNSUPPORTED: configuration not built";
    case UF_ERR_CAPACITY: return "UF_ERR_CAPACITY: window or pool full";
    case UF_ERR_EMPTY: return "UF_ERR_EMPTY: not enough chunks";
    case UF_ERR_HIP: return "UF_ERR_HIP: HIP runtime error";
    default: return "unknown status";
  }
}

const char* uf_last_error(void) { return g_last_error; }

}  // extern "C"
