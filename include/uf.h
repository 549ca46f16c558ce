/*
 * uf.h -- C ABI of the MI355X (gfx950) block-sparse chunk-causal attention path.
 *
 * The operation (Ultra Flash, arXiv 2606.09150, Sec. 2.3.1 (block-sparse causal
 * attention), Eq. 4, and Sec. 2.3.2 (dynamic cache management) (iii)):
 * a video is generated chunk by chunk; every attention layer keeps a KV cache
 * of earlier chunks (a compact window of a few chunks, App. C).
 * The current chunk's queries attend, with scaled softmax attention, over the
 * window's earlier chunks plus the current chunk (the temporal causal mask is
 * chunk-granular: no token-level triangle inside a chunk), restricted per
 * (head, query tile) to a kept subset of key tiles (the block mask of Eq. 4,
 * executed by a block-sparse kernel that skips every other tile).
 *
 * Entry points, in the order one chunk uses them:
 *   uf_kv_evict                 drop the oldest non-pinned chunks (host metadata)
 *   uf_kv_append                copy the current chunk's K and V into a free slot
 *   uf_build_tile_lists         per (b, h, query tile) keep lists of key tiles
 *                               (seeded Bernoulli stand-in), or
 *   uf_build_topk_lists         the same lists by content-adaptive top-k (Eq. 4)
 *   uf_sparse_causal_attn_fwd   attention of the current chunk's queries
 *   uf_sparse_causal_attn_bwd   its gradients (dQ, dK, dV)
 *
 * Conventions
 *   - bf16 tensors are raw IEEE bfloat16 bit patterns (uint16).
 *   - Q, K, V, O are [B, L, H, D] contiguous, D fastest, L = chunk_tokens.
 *   - Pointers named d_* are device pointers; the caller allocates and owns
 *     every device buffer (pool, Q, K, V, O, LSE, lists).  The library owns only
 *     the host-side handle; it never allocates device memory and never
 *     synchronises a stream.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *     device work is enqueued asynchronously on it; ring metadata changes at
 *     enqueue time.  Work on other streams must be ordered by the caller.
 *   - Every call returns a status code: UF_OK (0) or a negative UF_ERR_*.
 *     Nothing aborts, throws or prints.  On error the handle is unchanged and
 *     uf_last_error() describes the failure (thread-local text).
 *   - A handle is not thread-safe; distinct handles are independent.
 */
#ifndef UF_H
#define UF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define UF_OK               0
#define UF_ERR_ARG         (-1)  /* null/misaligned pointer, bad size or value   */
#define UF_ERR_UNSUPPORTED (-2)  /* valid but not built: head_dim != 128, tile not 64/128 */
#define UF_ERR_CAPACITY    (-3)  /* append into a full window; pool too small     */
#define UF_ERR_EMPTY       (-4)  /* evict more than evictable; work on no chunk   */
#define UF_ERR_HIP         (-5)  /* a HIP launch failed; uf_last_error() has text */

/* ---- flags (uf_kv_desc.flags) ----------------------------------------- */
#define UF_F_DRYRUN     1u  /* metadata only: no device work is enqueued, device
                               pointers are not dereferenced (host testing)  */
#define UF_F_POISON_PAD 2u  /* fill padding rows of partial tiles with bf16 9984.0
                               instead of 0 (checks that padding never counts) */

#define UF_MAX_CHUNKS 64    /* largest window capacity */
#define UF_MAX_SPLIT  64    /* largest split-KV slice count */

typedef struct uf_kv uf_kv; /* opaque host-side handle of one KV window */

/* Window description.  The window holds at most max_chunks chunks of
 * chunk_tokens tokens each, for batch x heads heads of dimension head_dim. */
typedef struct {
  int32_t batch;        /* B >= 1 */
  int32_t heads;        /* H >= 1 */
  int32_t head_dim;     /* D; must be 128 */
  int32_t chunk_tokens; /* L >= 1: frames * grid_h * grid_w tokens per chunk */
  int32_t tile;         /* T in {64, 128}: query tile = key tile = page rows */
  int32_t max_chunks;   /* 1 .. UF_MAX_CHUNKS, pinned chunk and current one included */
  int32_t pin_sink;     /* 1: the first appended chunk is never evicted */
  uint32_t flags;       /* UF_F_* */
} uf_kv_desc;

/* Keep rule for uf_build_tile_lists.  For query tile i of head (b, h) and key
 * tile t of the window chunk c:
 *   kept  if c is the pinned chunk and keep_sink,
 *   kept  if c is the current (most recently appended) chunk and keep_current,
 *   else  kept iff (x >> 32) < thr, where x = seed and, for each field f of
 *         (b, h, seq(current), i, seq(c), t) in turn, x = splitmix64(x ^ f);
 *         thr = 2^32 when p_prior >= 1, else floor(p_prior * 2^32) in double.
 * splitmix64(z): z += 0x9E3779B97F4A7C15, then z ^= z>>30, z *= 0xBF58476D1CE4E5B9,
 * z ^= z>>27, z *= 0x94D049BB133111EB, z ^= z>>31 (mod 2^64; Steele, Lea and
 * Flood, OOPSLA 2014).  This seeded Bernoulli rule stands in for the paper's
 * content-adaptive top-k of Eq. 4 (not part of the paper).  seq() are append
 * sequence numbers, so the lists depend only on the window's logical content. */
typedef struct {
  uint64_t seed;
  double p_prior;       /* in [0, 1]; 1 keeps every tile (dense) */
  int32_t keep_sink;    /* 0 or 1 */
  int32_t keep_current; /* 0 or 1 */
  int32_t local_r;      /* 0: no local mask; odd r >= 1: intersect with M_local
                           (needs block geometry, see uf_kv_set_block_geom) */
  int32_t reserved;     /* must be 0 */
} uf_keep_rule;

/* Content-adaptive top-k rule for uf_build_topk_lists (Sec. 2.3.1 (b), Eq. 4).
 * For query tile i of head (b, h) every key tile j of the window gets the score
 *   s(i, j) = qm(i) . km(j)
 * where qm(i) is the mean of the valid query tokens of tile i and km(j) the
 * mean of the valid key tokens of tile j (the block-mean pooling of Eq. 4; the
 * softmax and the factor 1/sqrt(d) of Eq. 4 are monotone and leave the ranking
 * unchanged).  Tiles of the pinned chunk (keep_sink) and of the current chunk
 * (keep_current) are kept without ranking; of the other tiles the `budget`
 * with the highest scores are kept, equal scores going to the lower logical
 * index.  Arithmetic is IEEE float32 in a fixed order: a mean is the
 * sequential sum over tokens in token order divided once by the valid count;
 * a score adds the rounded products qm[d]*km[d] in order of d, without fused
 * multiply-add; scores are compared as the unsigned key (bits of s with all
 * bits flipped when the sign is set, else with the sign bit set), which orders
 * float32 like the real line.  uf_topk_budget gives Eq. 10's budget. */
typedef struct {
  int32_t budget;       /* k >= 0: ranked tiles kept per row (all if k >= candidates) */
  int32_t keep_sink;    /* 0 or 1 */
  int32_t keep_current; /* 0 or 1 */
  int32_t local_r;      /* 0: no local mask; odd r >= 1: intersect the kept set
                           with M_local (needs block geometry) */
} uf_topk_rule;

typedef struct {
  int32_t n_live;     /* chunks in the window */
  int32_t nq_tiles;   /* NT = ceil(L / T): query tiles = key tiles per chunk */
  int32_t nk_tiles;   /* n_live * NT logical key tiles */
  int32_t tail_valid; /* valid tokens of each chunk's last tile, L - (NT-1)*T */
  int64_t first_seq;  /* seq of logical position 0, -1 if empty */
  int64_t last_seq;   /* seq of the current chunk, -1 if empty */
  int32_t has_sink;   /* 1 if logical position 0 is the pinned chunk */
  int32_t nk_cap;     /* max_chunks * NT: row capacity of the lists */
} uf_kv_info;

/* Device list buffer layout (all offsets in bytes from d_lists; R = B*H*NT rows,
 * row (b, h, i) = (b*H + h)*NT + i):
 *   counts  int32 [R]               kept key tiles of the row
 *   idx     int32 [R][nk_cap]       kept logical key tiles, ascending, then -1
 *   mask    uint32[R][mask_words]   bit j%32 of word j/32 set iff tile j kept
 *   scratch float [R][D]            working memory of uf_build_topk_lists (the
 *                                   pooled queries); contents unspecified
 * Logical key tile j is tile j % NT of the chunk at logical position j / NT;
 * logical order is [pinned chunk][oldest earlier .. newest earlier][current]. */
typedef struct {
  size_t counts_offset;
  size_t idx_offset;
  size_t mask_offset;
  size_t scratch_offset;
  size_t total_bytes;
  int32_t rows;
  int32_t nk_cap;
  int32_t mask_words;
  int32_t reserved;
} uf_lists_layout;

/* Pool bytes the window needs: max_chunks * B * H * NT pages of 4*T*D bytes,
 * then as many pooled keys of D float32 each (4*D bytes).
 * Page of (slot s, b, h, tile t) starts at ((((s*B + b)*H + h)*NT + t) * 4*T*D);
 * it holds K (row r = token t*T + r of the chunk), then V transposed (row d =
 * dimension d), both bf16, T*D elements each.  T = 128: both are stored as two
 * blocks of 64 columns, one after the other: K as [2][T][64] (block j holds
 * dimensions 64j..64j+63 of every key), V^T as [2][D][64] (block j holds keys
 * 64j..64j+63 of every dimension).  T = 64: K as [T][D] and V^T as [D][T].
 * In V^T the keys of each group of 16 are stored with bits 2 and 3 of the key
 * index swapped (column p of a block holds key
 * (p & ~12) | ((p & 4) << 1) | ((p & 8) >> 1) of that block).  Rows past the
 * chunk end are 0 (9984.0 under UF_F_POISON_PAD).  The pooled key of the same page, the float32
 * mean of its valid K rows (the key pooling of Eq. 4, written by append), starts
 * at max_chunks*B*H*NT*4*T*D + ((((s*B + b)*H + h)*NT + t) * 4*D).
 * Errors: UF_ERR_ARG, UF_ERR_UNSUPPORTED. */
int uf_kv_pool_bytes(const uf_kv_desc* desc, size_t* bytes);

/* Create a handle over a caller-owned pool (256-byte aligned, >= pool bytes).
 * The pool must outlive the handle; its contents are written by append only.
 * Errors: UF_ERR_ARG (null, misaligned, bad field), UF_ERR_UNSUPPORTED,
 * UF_ERR_CAPACITY (pool_bytes too small). */
int uf_kv_create(const uf_kv_desc* desc, void* d_pool, size_t pool_bytes, uf_kv** out);

/* Destroy a handle (host memory only).  NULL is accepted. */
int uf_kv_destroy(uf_kv* kv);

/* Append the current chunk (Alg. 3, inference: the SR DiT attends over its KV
 * cache plus the new chunk): copy K and V [B, L, H, D] bf16 (16-byte aligned)
 * into the pages of a free slot; it becomes the current chunk with the next
 * sequence number.  Errors: UF_ERR_ARG, UF_ERR_CAPACITY (window full), UF_ERR_HIP. */
int uf_kv_append(uf_kv* kv, const void* d_k, const void* d_v, void* stream);

/* Refresh the current chunk in place (Sec. 2.3.2 (ii), adaptive cache
 * refresh: the KV entries of the newest chunk are recomputed and replace the
 * ones appended from the last denoising step): copy K and V [B, L, H, D] bf16
 * (16-byte aligned) over the current chunk's pages and pooled keys.  Its
 * sequence number and logical position do not change, so Bernoulli lists are
 * unchanged and top-k lists must be rebuilt.  Reads of the old pages already
 * enqueued on the same stream happen first.  Errors: UF_ERR_ARG, UF_ERR_EMPTY
 * (no chunk), UF_ERR_HIP. */
int uf_kv_replace_newest(uf_kv* kv, const void* d_k, const void* d_v, void* stream);

/* 3-D block tiling of a chunk's token grid (Sec. 2.3.1 (a): the (t, h, w) grid
 * divided into non-overlapping (bt, bh, bw) blocks; (2, 8, 8) in the paper).
 * A chunk of `frames` latent frames on a grid_h x grid_w grid has blocks
 * (ceil(frames/bt), ceil(grid_h/bh), ceil(grid_w/bw)) in raster order (block
 * time, block row, block column).  In block order a chunk holds one tile of
 * bt*bh*bw rows per block: the block's valid tokens in raster (t, h, w) order,
 * then padding rows that count as no token.  With block geometry the local
 * window M_local(r) keeps key block j for query block i iff their block rows
 * and block columns differ by at most r/2 (integer division), in every chunk
 * and at every block time; it is intersected with the keep rule (forced
 * tiles included), as Eq. 4 intersects the content mask with the structural
 * ones. */
typedef struct {
  int32_t frames, grid_h, grid_w;
  int32_t bt, bh, bw;
} uf_block_geom;

#define UF_MAX_BLOCKS 2048  /* blocks per chunk under block geometry */

/* Tokens of a chunk in block order (blocks * bt*bh*bw) and its block count.
 * Errors: UF_ERR_ARG (null, non-positive field), UF_ERR_UNSUPPORTED (more
 * than UF_MAX_BLOCKS blocks). */
int uf_block_geom_tokens(const uf_block_geom* g, int32_t* padded_tokens, int32_t* n_blocks);

/* Give an empty window block geometry: its tiles become blocks (tile must be
 * bt*bh*bw and chunk_tokens the padded block-order length); append, the list
 * builders and attention then count a tile's valid rows from the geometry and
 * the rules may use M_local.  K, V and Q are passed in block order (see
 * uf_block_permute).  Errors: UF_ERR_ARG (bad geometry, mismatched tile or
 * chunk length, window not empty), UF_ERR_UNSUPPORTED (too many blocks). */
int uf_kv_set_block_geom(uf_kv* kv, const uf_block_geom* g);

/* Reorder [batch, tokens, heads, head_dim] bf16 rows between raster order
 * (frames*grid_h*grid_w tokens) and block order (padded block-order tokens):
 * inverse = 0 writes block order from raster (padding rows zero), inverse = 1
 * writes raster order from block order (padding rows dropped).  Buffers
 * 16-byte aligned, not overlapping; head_dim must be 128.  Errors: UF_ERR_ARG,
 * UF_ERR_UNSUPPORTED, UF_ERR_HIP. */
int uf_block_permute(const uf_block_geom* g, int32_t batch, int32_t heads, int32_t head_dim,
                     const void* d_src, void* d_dst, int32_t inverse, void* stream);

/* Drop the n oldest chunks that are not pinned (Sec. 2.3.2 (iii): a compact
 * cache window).  Host metadata only: the freed slot is rewritten by a later
 * append, which the stream orders after already-enqueued reads on that same
 * stream.  n = 0 is a no-op.  Errors: UF_ERR_ARG (n < 0), UF_ERR_EMPTY (fewer
 * than n evictable chunks). */
int uf_kv_evict(uf_kv* kv, int32_t n_chunks);

/* Window state.  Errors: UF_ERR_ARG. */
int uf_kv_get_info(const uf_kv* kv, uf_kv_info* info);

/* Slot and sequence number of logical position pos (0 <= pos < n_live).
 * Errors: UF_ERR_ARG. */
int uf_kv_logical(const uf_kv* kv, int32_t pos, int32_t* slot, int64_t* seq);

/* Layout and size of the list buffer.  Errors: UF_ERR_ARG. */
int uf_tile_lists_layout(const uf_kv* kv, uf_lists_layout* layout);
int uf_tile_lists_bytes(const uf_kv* kv, size_t* bytes);

/* Build the keep lists of the current window under `rule` into d_lists
 * (256-byte aligned, >= uf_tile_lists_bytes).  Valid until the next append or
 * evict.  Errors: UF_ERR_ARG, UF_ERR_EMPTY (no chunk), UF_ERR_HIP. */
int uf_build_tile_lists(const uf_kv* kv, const uf_keep_rule* rule, void* d_lists,
                        size_t bytes, void* stream);

/* Build the keep lists of the current window under the top-k `rule` from the
 * current chunk's queries d_q [B, L, H, D] bf16 (16-byte aligned) into d_lists
 * (same layout and validity as uf_build_tile_lists).  The ranked candidates of
 * a row must number at most 16384.  Errors: UF_ERR_ARG, UF_ERR_EMPTY (no
 * chunk), UF_ERR_UNSUPPORTED (too many candidates), UF_ERR_HIP. */
int uf_build_topk_lists(const uf_kv* kv, const void* d_q, const uf_topk_rule* rule,
                        void* d_lists, size_t bytes, void* stream);

/* Eq. 10's budget: max(k_min, floor(rho * seq_len / seq_ref * n_blocks)) in
 * double, clamped to int32.  Errors: UF_ERR_ARG (null out, rho < 0 or not
 * finite, seq_ref < 1, negative counts). */
int uf_topk_budget(double rho, int64_t seq_len, int64_t seq_ref, int64_t n_blocks, int32_t k_min,
                   int32_t* budget);

/* Block-sparse chunk-causal attention forward (Eq. 4 mask semantics): for each
 * (b, h) and query row r of the current chunk in query tile i,
 *   O[b,r,h,:] = sum_c softmax_c(scale * q.k_c) v_c over the tokens c of the
 *   kept key tiles of row (b, h, i) (padding excluded), and
 *   LSE[b,h,r] = natural log of sum_c exp(scale * q.k_c).
 * A row with no kept tile gives O = 0 and LSE = -inf.  q, o: [B, L, H, D] bf16,
 * 16-byte aligned; lse: [B, H, L] fp32 or NULL; d_lists as built by
 * uf_build_tile_lists for the current window (entries naming a tile outside
 * the window are skipped).  scale must be positive and finite, with
 * scale*log2(e) a normal float (else UF_ERR_ARG).  Computes in fp32 with bf16
 * MFMA products; O is rounded to nearest even.  Errors: UF_ERR_ARG,
 * UF_ERR_EMPTY, UF_ERR_HIP. */
int uf_sparse_causal_attn_fwd(const uf_kv* kv, const void* d_q, const void* d_lists,
                              float scale, void* d_o, float* d_lse, void* stream);

/* Split-KV attention (for windows whose rows are too few to fill the GPU):
 * the same operation as uf_sparse_causal_attn_fwd, with the kept-tile list of
 * every row cut into n_split contiguous slices (slice s takes entries
 * [s*count/n_split, (s+1)*count/n_split)) that separate workgroups attend;
 * each slice leaves its unnormalised output, running offset and row sum in
 * d_work, and a merge combines them by the same log-sum-exp rescaling as the
 * online softmax.  d_work (16-byte aligned, >= uf_attn_split_work_bytes) is
 * caller-owned scratch, overwritten.  Both tile sizes.  Results equal those
 * of uf_sparse_causal_attn_fwd up to float rounding order.  Errors:
 * UF_ERR_ARG, UF_ERR_EMPTY, UF_ERR_HIP. */
int uf_attn_split_work_bytes(const uf_kv* kv, int32_t n_split, size_t* bytes);
int uf_sparse_causal_attn_fwd_split(const uf_kv* kv, const void* d_q, const void* d_lists, float scale,
                                    void* d_o, float* d_lse, int32_t n_split, void* d_work,
                                    size_t work_bytes, void* stream);

/* Split-KV of the rows of the last, partly filled round only.  With one
 * workgroup per compute unit a window of R rows runs in ceil(R / n_cu) rounds;
 * when the last round is partly empty (444 rows on 256 CUs: the second round
 * leaves 68 CUs idle), cutting only its rows into slices that fill the
 * compute units shortens the launch.  uf_sparse_causal_attn_fwd_split_rows
 * runs rows 0 .. split_from-1 whole and cuts every later row into n_split
 * slices as uf_sparse_causal_attn_fwd_split does (split_from = 0: every row,
 * which is that entry point; split_from = rows: none), with a merge of the
 * split rows; d_work (16-byte aligned, >= uf_attn_split_rows_work_bytes, may
 * be NULL when no row is split) is caller-owned scratch, overwritten.
 * uf_attn_tail_plan picks split_from and n_split for a device with n_cu compute
 * units, counting C = n_cu resident workgroups (one per compute unit with either
 * tile size): split_from = C * floor(R / C) and the n_split in 2..8
 * (in 2..min(64, C / R) when R < C), at most the window's key tiles, that
 * makes the last round shortest, in row-times
 * ceil((R - split_from) * n_split / C) * (1 / n_split + 9 / nk) + 12 / nk
 * (nk = the window's key tiles: a slice's fixed cost and the merge launch,
 * measured, in key tiles of work); it returns split_from = R and
 * n_split = 1 (no split) when R is a multiple of C or when the saving is
 * under a fifth of a row-time or under 16 key tiles of one row's work.  Results equal those of uf_sparse_causal_attn_fwd
 * up to float rounding order.  Errors: UF_ERR_ARG, UF_ERR_EMPTY, UF_ERR_HIP. */
int uf_attn_tail_plan(const uf_kv* kv, int32_t n_cu, int32_t* split_from, int32_t* n_split);
int uf_attn_split_rows_work_bytes(const uf_kv* kv, int32_t split_from, int32_t n_split, size_t* bytes);
int uf_sparse_causal_attn_fwd_split_rows(const uf_kv* kv, const void* d_q, const void* d_lists, float scale,
                                         void* d_o, float* d_lse, int32_t split_from, int32_t n_split,
                                         void* d_work, size_t work_bytes, void* stream);

/* Backward of uf_sparse_causal_attn_fwd (the student's training side of
 * Sec. 2.3.1: gradients through the same Eq. 4 mask).  With p = exp(scale*q.k
 * - LSE) over the kept keys of each row, delta = <dO, O> per row and
 * dS = p * (dO.v - delta):
 *   dQ = scale * sum_c dS_c k_c,  dK_c = scale * sum_r dS_rc q_r,
 *   dV_c = sum_r p_rc dO_r
 * (keys of no kept tile and padding rows get zero).  d_q, d_o (the forward's
 * output), d_do: [B, L, H, D] bf16, 16-byte aligned; d_lse [B, H, L] fp32, the
 * forward's LSE for the same window, queries and d_lists (both the index and
 * the mask sections are read, so they must come from one list build).
 * Outputs, fp32, 16-byte aligned, fully overwritten: d_dq [B, L, H, D];
 * d_dk, d_dv [n_live, B, L, H, D] in logical chunk order (position 0 first).
 * d_work (16-byte aligned, >= uf_attn_bwd_work_bytes) is caller-owned scratch,
 * overwritten.  Deterministic (no atomics).  Both tile sizes (at most 2,048
 * query tiles per chunk), head_dim 128.  Errors: UF_ERR_ARG,
 * UF_ERR_UNSUPPORTED (more query tiles), UF_ERR_EMPTY, UF_ERR_HIP. */
int uf_attn_bwd_work_bytes(const uf_kv* kv, size_t* bytes);
int uf_sparse_causal_attn_bwd(const uf_kv* kv, const void* d_q, const void* d_o, const void* d_do,
                              const float* d_lse, const void* d_lists, float scale, float* d_dq,
                              float* d_dk, float* d_dv, void* d_work, size_t work_bytes, void* stream);

/* No-allocation backward, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving or training loops, harnesses
 * that forbid allocation): the same operation, arguments, outputs and errors
 * as uf_sparse_causal_attn_bwd, without the workspace.  Its query-tile
 * records (the 66,560 bytes per list row that uf_attn_bwd_work_bytes counts)
 * live in a device array inside the library, UF_BWD_SCRATCH_BYTES on every GPU
 * it runs on, held from the first call on that GPU until the process ends.
 * Needs B*H*NT*66560 <= UF_BWD_SCRATCH_BYTES, i.e. at most 1,008 list rows
 * (query tiles over all heads), else UF_ERR_CAPACITY.  Every call on one GPU
 * uses the same array and leaves the last call's records in it (each call
 * rewrites every record it reads first, so nothing needs clearing): calls that
 * overlap in time on one GPU (other streams, or other threads without
 * ordering) race and give wrong results; calls ordered on one stream are safe.
 * The first call on a GPU looks the array's address up (no allocation); no
 * call allocates or frees device or pinned memory.  Errors: as
 * uf_sparse_causal_attn_bwd, plus UF_ERR_CAPACITY. */
#define UF_BWD_SCRATCH_BYTES ((size_t)64 << 20)
int uf_sparse_causal_attn_bwd_noalloc(const uf_kv* kv, const void* d_q, const void* d_o, const void* d_do,
                                      const float* d_lse, const void* d_lists, float scale, float* d_dq,
                                      float* d_dk, float* d_dv, void* stream);

/* Static text of a status code. */
const char* uf_status_string(int status);

/* Thread-local description of the last error returned on this thread. */
const char* uf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* UF_H */
