/*
 * wsk.h -- C ABI of a partitioned KV cache for CPU-GPU split decode attention
 * on AMD Instinct MI355X (gfx950).
 *
 * The cache follows the format of Yu, Dong, Liao, "Physically Partitioned
 * KVCache Format for CPU-GPU Load Balancing in MoE Inference":
 *
 *   - Sec. 3 and Sec. 4.3 (i): every cached byte gets its one physical home
 *     when it is written, and placed data never moves afterwards.  A
 *     sequence's positions [0, s) go to the CPU partition (pageable host
 *     memory, read in place by the CPU engine), [s, load_end) to the load
 *     region (pinned host memory in the GPU's slot layout, streamed to the
 *     GPU through a ping-pong pair of HBM buffers), and later positions to
 *     the GPU pool in HBM; s and load_end are fixed when the sequence is
 *     opened.  By default load_end = s and the GPU side is HBM-resident.
 *   - Sec. 4.2: decode rows are appended to the GPU pool (the D-window);
 *     wsk_flush evicts whole batches of D rows from it to the CPU partition
 *     or the load region, where they stay.
 *   - Sec. 4.1: each partition is made of fixed-size blocks of block_tokens
 *     tokens on an absolute grid (block k holds positions [k*Bk, (k+1)*Bk)).
 *     A block straddling s has a slot in both pools, each holding only its
 *     own side's positions.
 *   - Sec. 4.3: the interface is a PartitionSpec plus init / append / views
 *     / flush.  The GPU side additionally attends its own range and merges
 *     partial results (Sec. 4.2, last paragraph; Sec. 5.1).
 *
 * Conventions for every call:
 *   - The return value is a status: WSK_OK (0) or a negative WSK_E* code.
 *     wsk_last_error() returns a message for the calling thread's last
 *     failure.  No C++ exception crosses this boundary.
 *   - A failed call changes no cache state and enqueues no GPU work, except
 *     WSK_EHIP, which reports a HIP runtime failure after the fact.
 *   - "stream" is a hipStream_t passed as void* (NULL = the legacy default
 *     stream).  GPU work is enqueued on it in call order; results in device
 *     memory are ready when the stream reaches that point.
 *   - bf16 values are raw IEEE bfloat16 bits (uint16_t storage).
 *   - A cache is not thread-safe: serialise calls on one cache.
 */
#ifndef WSK_H
#define WSK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define WSK_OK 0
#define WSK_EINVAL (-1) /* malformed argument or spec                         */
#define WSK_ENOMEM (-2) /* a block pool (or a host allocation) is exhausted   */
#define WSK_ERANGE (-3) /* a position or range outside what the call allows   */
#define WSK_EHIP (-4)   /* the HIP runtime reported an error                  */
#define WSK_ESTATE (-5) /* wrong state: sequence not open / already open, or
                           a GPU call on a cache created without a device      */

#define WSK_KIND_GQA 0 /* per-head K and V rows, grouped-query attention     */
#define WSK_KIND_MLA 1 /* one compressed latent row per token (MLA)          */

#define WSK_PART_CPU 0
#define WSK_PART_GPU 1  /* the GPU pool in HBM                                */
#define WSK_PART_LOAD 2 /* the pinned load region, streamed to the GPU        */

#define WSK_LAYOUT_ROWS 0    /* token-major rows                               */
#define WSK_LAYOUT_TILED64 1 /* GQA GPU pool: 64-token tiles in matrix-core order */
#define WSK_LAYOUT_MLA32 2   /* MLA GPU pool: 32-token tiles in matrix-core order */

/* Largest number of query heads one KV head may serve in a GQA cache.       */
#define WSK_MAX_GROUP 64

/*
 * PartitionSpec (Sec. 4.3): the physical layout of one layer's cache.  The
 * paper's spec also carries the roofline parameters of its split policy;
 * this library takes the split per sequence instead (wsk_seq_open).
 *
 *   kind               WSK_KIND_GQA or WSK_KIND_MLA
 *   n_q_heads          query heads (MLA: heads sharing the latent)
 *   n_kv_heads         GQA: KV heads, dividing n_q_heads with
 *                      n_q_heads / n_kv_heads <= WSK_MAX_GROUP; MLA: 1
 *   head_dim           GQA: K/V width, must be 128.  MLA: ignored.
 *   latent_dim         MLA: compressed latent width, must be 512.  GQA: 0.
 *   rope_dim           MLA: decoupled RoPE key width, must be 64.  GQA: 0.
 *   block_tokens       tokens per block: 64, 128 or 256 (each divides the
 *                      paper's eviction batch of 256, Sec. 4.2)
 *   max_seqs           sequence ids are 0 .. max_seqs-1
 *   max_seq_len        positions per sequence, >= 1
 *   device_pool_blocks slots in the GPU pool (HBM), >= 0
 *   host_pool_blocks   slots in the CPU pool (pageable host memory), >= 0
 *   softmax_scale      multiplier of q.k before the softmax, finite and > 0
 *   evict_tokens       D, the eviction batch of wsk_flush (Sec. 4.2): a
 *                      multiple of block_tokens, or 0 (no eviction); a
 *                      device cache with D > 0 pins, at init, a host bounce
 *                      for one batch of every sequence (at most 64 MB)
 *   load_arena_blocks  load-region slots pinned by one host allocation; the
 *                      region is pinned arena by arena as it fills, one
 *                      arena ahead of use (Sec. 4.3 end, Sec. 5)
 *   pingpong_blocks    slots of each of the two HBM ping-pong buffers that
 *                      the load region is streamed through (Sec. 4.2)
 *   load_pool_blocks   slots of the load region, >= 0; 0 = no load region
 *                      (then load_arena_blocks and pingpong_blocks are 0),
 *                      else load_arena_blocks > 0 and pingpong_blocks > 0
 *
 * Slot layouts (bf16).  Each partition's layout is fixed by the format for
 * the engine that reads it (Sec. 4.3 (ii)):
 *   GQA, CPU pool  slot = [n_kv_heads][2][block_tokens][head_dim]
 *                  (per head: K rows, then V rows; token-major)
 *   GQA, GPU pool  slot = [n_kv_heads][block_tokens / 64 tiles][K: 1024 | V: 1024]
 *                  16-byte pieces, each piece 8 bf16, in the order the GPU
 *                  kernel's matrix-core lanes read them (WSK_LAYOUT_TILED64):
 *                  token t of a tile (0..63), dim d (0..127):
 *                    K: piece (4*mt + d/32)*64 + 16*((d%32)/8) + nk, elem d%8,
 *                       mt = 2*(t/32) + (t%8)/4,  nk = 4*((t%32)/8) + t%4
 *                    V: piece (2*(d/16) + t/32)*64 + 16*((t%32)/8) + d%16,
 *                       elem t%8
 *   MLA, CPU pool  slot = [block_tokens][latent_dim + rope_dim]  (latent | rope)
 *   (The load region's slots have the GPU pool's layout, so that a DMA
 *   lands them ready for the GPU kernels.)
 *   MLA, GPU pool  slot = [block_tokens / 32 tiles][2304 16-byte pieces]
 *                  (WSK_LAYOUT_MLA32); piece c (dims 8c..8c+7, c = 0..71) of
 *                  token u of a tile (0..31) is piece
 *                    (2*(c/4) + (u/4)%2)*64 + 16*(c%4) + 4*(u/8) + u%4
 */
typedef struct wsk_partition_spec {
    int32_t kind;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t latent_dim;
    int32_t rope_dim;
    int32_t block_tokens;
    int32_t max_seqs;
    int32_t max_seq_len;
    int32_t reserved; /* must be 0 */
    int64_t device_pool_blocks;
    int64_t host_pool_blocks;
    float softmax_scale;
    int32_t evict_tokens;
    int32_t load_arena_blocks;
    int32_t pingpong_blocks;
    int64_t load_pool_blocks;
} wsk_partition_spec;

typedef struct wsk_cache wsk_cache;

/* Where one cached position lives (wsk_route). */
typedef struct wsk_loc {
    int32_t part;          /* WSK_PART_CPU, WSK_PART_GPU or WSK_PART_LOAD */
    int32_t logical_block; /* pos / block_tokens                      */
    int32_t slot;          /* slot index in that partition's pool     */
    int32_t offset;        /* pos % block_tokens: row within the slot */
} wsk_loc;

/*
 * Zero-copy view of one partition of one sequence (Sec. 4.3 (iii)).
 * For token p of the partition (start <= p < end) and KV head g, let
 *   head = (char*)pool + table[p / block_tokens] * slot_bytes + g * head_bytes.
 * layout WSK_LAYOUT_ROWS: the K row (or MLA row) is at
 *   head + (p % block_tokens) * row_bytes,
 *   and (GQA) the V row at head + v_bytes + (p % block_tokens) * row_bytes.
 * layout WSK_LAYOUT_TILED64 (GQA GPU pool): tile k = (p % block_tokens) / 64
 *   starts at head + k * 32768; its K pieces follow, then its V pieces at
 *   + 16384, placed as described for the slot layout above.
 * layout WSK_LAYOUT_MLA32 (MLA GPU pool): tile k = (p % block_tokens) / 32
 *   starts at head + k * 36864, pieces placed as described above.
 * CPU views hold host addresses; GPU views hold device addresses (the table
 * too).  The pointers are borrowed: they stay valid until wsk_destroy,
 * because placed blocks never move (Sec. 4.2).
 */
typedef struct wsk_view {
    void *pool;
    const int32_t *table; /* this sequence's row: slot per logical block, -1 = none */
    int64_t slot_bytes;
    int64_t head_bytes;
    int64_t v_bytes;
    int64_t row_bytes;
    int32_t start, end;   /* CPU: [0, min(s, L)); GPU: the D-window [min(w, L), L);
                             later CPU segments (wsk_seq_segments) use the same table */
    int32_t block_tokens;
    int32_t is_device;
    int32_t layout;       /* WSK_LAYOUT_ROWS, WSK_LAYOUT_TILED64 or WSK_LAYOUT_MLA32 */
    int32_t reserved;
} wsk_view;

/* Message of the calling thread's last failure ("" if none). */
const char *wsk_last_error(void);

/*
 * Validate *spec and build a cache (Sec. 4.3 "init").  device >= 0 selects
 * the HIP device that owns the GPU pool; both pools and the block tables
 * are allocated here, once, and zero-filled.  device = -1 builds a
 * host-only cache that never calls HIP: routing, wsk_reserve, wsk_route
 * and CPU views work; every call that moves data to or computes on the GPU
 * returns WSK_ESTATE.  The library owns the cache; free it with wsk_destroy.
 * Errors: EINVAL (spec), ENOMEM (host allocation), EHIP (device allocation).
 */
int wsk_init(const wsk_partition_spec *spec, int device, wsk_cache **out);

/* Free both pools and tables.  The caller must have synchronised every
 * stream that still uses the cache.  NULL is accepted. */
int wsk_destroy(wsk_cache *cache);

/* Copy of the cache's spec. */
int wsk_get_spec(const wsk_cache *cache, wsk_partition_spec *out);

/*
 * Open sequence seq with split s >= 0: positions p < s will live in the CPU
 * partition and p >= s in the GPU partition (the paper's sequence-dimension
 * split, Sec. 5.1, fixed at write time).  Errors: EINVAL (seq or s out of
 * range), ESTATE (already open).
 */
int wsk_seq_open(wsk_cache *cache, int32_t seq, int32_t split);

/*
 * Open seq with a load range: positions p < split go to the CPU partition,
 * split <= p < load_end to the load region (the paper's pinned load region,
 * Sec. 4.2), p >= load_end to the GPU pool (the D-window, where decode rows
 * are appended).  load_end >= split; a non-empty load range needs a load
 * region and load_end a multiple of block_tokens (so that every later block
 * of the GPU pool is whole).  wsk_seq_open(c, seq, s) is
 * wsk_seq_open_window(c, seq, s, s).  Errors: EINVAL, ESTATE.
 */
int wsk_seq_open_window(wsk_cache *cache, int32_t seq, int32_t split, int32_t load_end);

/* Close seq and return all its slots to the free sets (in-place block
 * reclamation at session end, Sec. 4.2).  Work already enqueued that reads
 * those slots must be ordered before any later write that reuses them.
 * Errors: EINVAL, ESTATE (not open). */
int wsk_seq_close(wsk_cache *cache, int32_t seq);

/* Current length L and split s of an open sequence. */
int wsk_seq_info(const wsk_cache *cache, int32_t seq, int32_t *length, int32_t *split);

/*
 * Routing decision only (Sec. 4.3 (i), "append is the routing decision"):
 * give positions [L, L+n) of seq their homes, taking slots lowest-free-first,
 * and set L += n, without writing data.  The rows hold whatever the slot held
 * before (zeros for never-used slots) until the caller fills them, e.g.
 * through wsk_views.  All-or-nothing: ENOMEM leaves the cache unchanged.
 * Errors: EINVAL (n < 0 or past max_seq_len), ESTATE, ENOMEM.
 */
int wsk_reserve(wsk_cache *cache, int32_t seq, int32_t n);

/*
 * Bulk write of positions [pos0, pos0+n) of seq (prefill routed in one shot,
 * Sec. 4.2): each row goes to its partition's pool.  pos0 must equal the
 * current length L.  k, v are HOST pointers, token-major:
 *   GQA  k, v: bf16 [n][n_kv_heads][head_dim]
 *   MLA  k:    bf16 [n][latent_dim + rope_dim], v must be NULL
 * CPU rows are copied with memcpy; GPU rows go host -> device through a
 * staging buffer and a scatter kernel on stream.  The call returns after the
 * data is in place (it synchronises stream), so k and v may be freed at once.
 * All-or-nothing for routing (ENOMEM changes nothing).
 * Errors: EINVAL, ESTATE, ERANGE (pos0 != L), ENOMEM, EHIP.
 */
int wsk_write(wsk_cache *cache, int32_t seq, int32_t pos0, int32_t n,
              const void *k, const void *v, void *stream);

/*
 * Decode append (Sec. 4.2: new entries join the GPU side at no transfer
 * cost): one new row at position L of each listed sequence, then L += 1.
 * seq_ids is a HOST array of n distinct open sequences; k_new, v_new are
 * DEVICE pointers, row i for seq_ids[i]:
 *   GQA  k_new, v_new: bf16 [n][n_kv_heads][head_dim]
 *   MLA  k_new:        bf16 [n][latent_dim + rope_dim], v_new NULL
 * (16-byte aligned).
 * Routing (slot allocation) happens on the host during the call; the copy
 * runs asynchronously on stream, and the inputs must stay valid until the
 * stream reaches it.  Every appended position must be in the GPU partition
 * (L >= s); rows below the split are written with wsk_write.
 * Errors: EINVAL (n <= 0, duplicate or bad ids), ESTATE, ERANGE (position
 * below the split or past max_seq_len), ENOMEM, EHIP.
 */
int wsk_append(wsk_cache *cache, int32_t n, const int32_t *seq_ids,
               const void *k_new, const void *v_new, void *stream);

/* Home of position pos of seq.  Errors: EINVAL, ESTATE, ERANGE (pos >= L). */
int wsk_route(const wsk_cache *cache, int32_t seq, int32_t pos, wsk_loc *out);

/* Zero-copy views of both partitions of seq (Sec. 4.3 "views").  Either
 * output pointer may be NULL.  The GPU view of a host-only cache has NULL
 * pool and table.  Errors: EINVAL, ESTATE. */
int wsk_views(const wsk_cache *cache, int32_t seq, wsk_view *cpu, wsk_view *gpu);

/*
 * Bytes of device workspace wsk_attend needs for the same sequences and
 * ranges (the split-KV chunk partials).  Same argument rules as wsk_attend.
 */
int wsk_attend_workspace(const wsk_cache *cache, int32_t n, const int32_t *seq_ids,
                         const int32_t *start, const int32_t *end, size_t *bytes);

/*
 * Decode attention over the GPU partition (the GPU engine of Sec. 5.1): for
 * each i < n, every query head of seq_ids[i] attends positions
 * [start[i], end[i]), which must lie in the GPU pool (the D-window):
 * min(w, L) <= start <= end <= L, where w is the window's start (w = s for
 * a sequence opened without a load range and never flushed; the load
 * region is attended by wsk_attend_gpu).  The output
 * is a normalised partial and its log-sum-exp (Sec. 4.2 last paragraph):
 *   O[i][h]   = sum_j softmax_j(scale * q.k_j) v_j
 *   LSE[i][h] = ln sum_j exp(scale * q.k_j)
 * An empty range gives O = 0, LSE = -inf and reads no KV.
 * Query head h reads KV head floor(h / (n_q_heads / n_kv_heads)).
 * seq_ids, start, end: HOST arrays (seq ids need not be distinct).
 * q, o, lse, ws: DEVICE pointers owned by the caller:
 *   GQA  q bf16 [n][n_q_heads][head_dim]       o fp32 [n][n_q_heads][head_dim]
 *   MLA  q bf16 [n][n_q_heads][latent+rope]    o fp32 [n][n_q_heads][latent_dim]
 *        (the absorbed query q_lat | q_rope)   (the latent output, before expansion)
 *   lse fp32 [n][n_q_heads] (natural log)
 *   ws   at least wsk_attend_workspace() bytes, 256-byte aligned
 *   q and o 16-byte aligned
 * Softmax and accumulation are fp32 from bf16 inputs.
 * Errors: EINVAL, ESTATE, ERANGE (range outside the GPU partition), EHIP.
 */
int wsk_attend(wsk_cache *cache, int32_t n, const int32_t *seq_ids,
               const int32_t *start, const int32_t *end, const void *q,
               float *o, float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * The two passes of wsk_attend, for callers that schedule or time them
 * apart.  Called with the same cache state, seq_ids, start, end and
 * workspace, wsk_attend_pass1 followed by wsk_attend_pass2 (o_x, lse_x NULL)
 * on the stream is wsk_attend:
 *   pass 1 attends every chunk of every range (split-KV: each range is cut
 *          into chunks of whole 64-token tiles spread over the GPU) and
 *          leaves each chunk's normalised partial O and LSE in ws;
 *   pass 2 merges the chunks of each (sequence, head) by their LSE into o
 *          and lse.
 * o_x, lse_x (DEVICE, both or neither; o_x 16-byte aligned): a partial over
 * other keys with the layout of o and lse, e.g. the CPU range's (O, LSE)
 * (Sec. 4.2, Sec. 5.1).  Given, pass 2 merges it in as one more chunk, so o
 * and lse are the LSE merge of the CPU and GPU partials, as wsk_attend
 * followed by wsk_merge would give (up to fp32 rounding order), in one
 * launch.  An empty GPU range then returns the other partial unchanged.
 * The workspace contents between the passes are private to the library.
 * Arguments, ownership and errors as for wsk_attend (pass 1 takes no o/lse,
 * pass 2 no q).
 */
int wsk_attend_pass1(wsk_cache *cache, int32_t n, const int32_t *seq_ids,
                     const int32_t *start, const int32_t *end, const void *q,
                     void *ws, size_t ws_bytes, void *stream);
int wsk_attend_pass2(wsk_cache *cache, int32_t n, const int32_t *seq_ids,
                     const int32_t *start, const int32_t *end,
                     const float *o_x, const float *lse_x, float *o,
                     float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * LSE merge of two partials over disjoint key sets (Sec. 4.2, Sec. 5.1),
 * row by row, on the GPU:
 *   m = max(lse_a, lse_b);  m = -inf  ->  O = 0, LSE = -inf
 *   otherwise w_x = exp(lse_x - m),  O = (w_a O_a + w_b O_b) / (w_a + w_b),
 *   LSE = m + ln(w_a + w_b)
 * All pointers are DEVICE pointers: o_* fp32 [rows][width], lse_* fp32
 * [rows]; o_a, o_b, o_out 16-byte aligned.  o_out/lse_out may alias o_b/lse_b
 * (or o_a/lse_a).  o_bf16, if not NULL, also receives O rounded to bf16
 * (nearest-even), [rows][width].
 * Errors: EINVAL (rows < 0, width <= 0 or width % 4 != 0), EHIP.
 */
int wsk_merge(int32_t rows, int32_t width, const float *o_a, const float *lse_a,
              const float *o_b, const float *lse_b, float *o_out, float *lse_out,
              uint16_t *o_bf16, void *stream);

/*
 * MLA query-side projection (Sec. 6.1, compressed-MLA variant): for each of
 * n tokens and H heads, q_lat[h] = W_UK[h]^T q_nope[h] with fp32
 * accumulation, rounded once to bf16 (nearest-even).  DEVICE pointers:
 *   q_nope bf16 [n][H][dn], w_uk bf16 [H][dn][dl],
 *   out: row (i, h) is written at out + (i*H + h) * out_stride elements
 *   (out_stride >= dl; pass latent+rope to fill the first dl elements of an
 *   attend query buffer in place).
 * Supported: dl % 64 == 0, 1 <= dn <= 256; w_uk 16-byte aligned.
 * Errors: EINVAL, EHIP.
 */
int wsk_mla_absorb(int32_t n, int32_t H, int32_t dn, int32_t dl, const uint16_t *q_nope,
                   const uint16_t *w_uk, uint16_t *out, int64_t out_stride, void *stream);

/*
 * MLA output-side expansion (Sec. 6.1): O[i][h] = W_UV[h]^T O_lat[i][h],
 * fp32 accumulation.  DEVICE pointers: o_lat fp32 [n][H][dl],
 * w_uv bf16 [H][dl][dv], o fp32 [n][H][dv].
 * Supported: dv % 64 == 0, 1 <= dl <= 1024; w_uv 16-byte aligned.
 * Errors: EINVAL, EHIP.
 */
int wsk_mla_expand(int32_t n, int32_t H, int32_t dl, int32_t dv, const float *o_lat,
                   const uint16_t *w_uv, float *o, void *stream);

/*
 * Block-sparse decode attention over the GPU side (Sec. 4.4): a block-level
 * selection (e.g. a top-k over blocks computed by the model) yields whole
 * blocks, and each query head of seq_ids[i] attends only the positions of
 * its selected logical blocks
 *   sel[sel_begin[i] .. sel_begin[i+1])      (sel_begin: n + 1 entries, [0] = 0)
 * that lie on the GPU side: in the GPU pool (the D-window [w, L)) or in the
 * load region.  A block holding s contributes its positions >= s, the block
 * holding L - 1 those < L.  Blocks must be distinct, in any order, each with
 * GPU-side positions; none selected gives O = 0, LSE = -inf.  Selected
 * GPU-pool blocks are read in place, through a compacted copy of their table
 * entries kept in ws.  Selected load-region blocks are gathered by the host,
 * one memcpy per block, into pinned staging and sent as one contiguous DMA
 * per ping-pong buffer (the gather of the next buffer overlaps the DMA of
 * the current one); the call returns when the last gather is done.
 * o_x, lse_x: optional partial to merge in, as for wsk_attend_pass2.
 * All of seq_ids, sel_begin, sel are HOST arrays; q, o_x, lse_x, o, lse, ws
 * DEVICE pointers laid out as for wsk_attend; ws of at least
 * wsk_attend_blocks_workspace() bytes.  Errors: EINVAL (malformed or
 * repeated selection), ERANGE (block without GPU-side positions), ESTATE,
 * EHIP.
 */
int wsk_attend_blocks_workspace(const wsk_cache *cache, int32_t n, const int32_t *seq_ids,
                                const int32_t *sel_begin, const int32_t *sel, size_t *bytes);
int wsk_attend_blocks(wsk_cache *cache, int32_t n, const int32_t *seq_ids,
                      const int32_t *sel_begin, const int32_t *sel, const void *q,
                      const float *o_x, const float *lse_x, float *o, float *lse,
                      void *ws, size_t ws_bytes, void *stream);

/*
 * In-place CPU attention over the CPU partition (the CPU engine of Sec. 5.1;
 * MLA: the latent variant of Sec. 6.1): for each i < n, every query head of
 * seq_ids[i] attends positions [start[i], end[i]), which must all be in the
 * CPU partition (the prefix [0, min(s, L)) and the batches wsk_flush moved
 * there).  Rows are read where they sit in the host pool, block by block
 * through the CPU block table (Sec. 4.3
 * (iii)); nothing is copied.  The result is the same normalised partial O
 * and natural-log LSE as wsk_attend's (O = 0, LSE = -inf for an empty
 * range), ready for the LSE merge with the GPU partial.
 * seq_ids, start, end, q, o, lse: HOST arrays; q, o, lse laid out as for
 * wsk_attend.  threads: host threads to use (<= 0: every hardware thread).
 * fp32 arithmetic from bf16 rows.  Synchronous: returns when done.  It
 * touches host memory only, so GPU work already enqueued keeps running
 * meanwhile; it must not overlap calls that change the cache.  Works on
 * host-only caches.  Errors: EINVAL, ESTATE, ERANGE.
 */
int wsk_cpu_attend(wsk_cache *cache, int32_t n, const int32_t *seq_ids,
                   const int32_t *start, const int32_t *end, const void *q,
                   float *o, float *lse, int32_t threads);

/*
 * wsk_cpu_attend over every CPU-partition position of each listed sequence
 * (the prefix [0, min(s, L)) and all batches flushed to the CPU): one
 * partial (O, LSE) per sequence.  Arguments as for wsk_cpu_attend.
 */
int wsk_cpu_attend_all(wsk_cache *cache, int32_t n, const int32_t *seq_ids, const void *q, float *o,
                       float *lse, int32_t threads);

/*
 * The GPU side of one decode step (Sec. 4.2): every query head of seq_ids[i]
 * attends all of the sequence's GPU-side positions -- the D-window [w, L)
 * in place in HBM, and the load-region positions streamed host -> device
 * through the two ping-pong buffers (Sec. 4.2: the buffers are allocated
 * once and overwritten in turn; each is refilled as soon as the kernels
 * reading it finish, so the DMA of one buffer overlaps the attention over
 * the other).  Runs of consecutive load slots travel as one DMA each.  The
 * chunk partials, plus o_x / lse_x when given (the CPU partial), are merged
 * into o / lse.  q, o_x, lse_x, o, lse, ws: DEVICE pointers laid out as for
 * wsk_attend; ws of at least wsk_attend_gpu_workspace() bytes, 256-byte
 * aligned.  The DMA runs on the cache's own copy stream, ordered after the
 * evictions of earlier wsk_flush calls; the kernels run on stream.
 * Returns after enqueueing.  Errors: EINVAL, ESTATE, EHIP.
 */
int wsk_attend_gpu_workspace(const wsk_cache *cache, int32_t n, const int32_t *seq_ids, size_t *bytes);
int wsk_attend_gpu(wsk_cache *cache, int32_t n, const int32_t *seq_ids, const void *q, const float *o_x,
                   const float *lse_x, float *o, float *lse, void *ws, size_t ws_bytes, void *stream);

/* wsk_attend_gpu as its two passes, so that the CPU engine can compute the
 * CPU partial while the load region streams (Sec. 4.2: the CPU and the GPU
 * attend at the same time, one join per step): pass 1 enqueues the
 * transfers and the attention kernels and leaves the partials in ws; pass 2,
 * called with the same sequences and no cache change in between, merges
 * them and o_x / lse_x into o / lse.  Arguments as for wsk_attend_gpu. */
int wsk_attend_gpu_pass1(wsk_cache *cache, int32_t n, const int32_t *seq_ids, const void *q, void *ws,
                         size_t ws_bytes, void *stream);
int wsk_attend_gpu_pass2(wsk_cache *cache, int32_t n, const int32_t *seq_ids, const float *o_x,
                         const float *lse_x, float *o, float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * One decode step of the GPU side (Sec. 4.2): the append of each listed
 * sequence's new row at position L (as wsk_append), then every query head
 * attends all its GPU-side positions [.., L] -- the new row included -- and
 * the result is merged with o_x / lse_x when given (as wsk_attend_gpu).
 * Same result as wsk_append followed by wsk_attend_gpu: pass 1 covers the
 * positions written before the call, and pass 2 scores the new row straight
 * from k_new (q . k_new), merges it as one more partial and stores it into
 * the GPU pool.  GQA without load-region positions: one kernel launch per 64
 * sequences, pass 2 done by the last workgroup of each (sequence, KV head,
 * head group) to finish its pass-1 chunk (counted with device-scope atomics
 * on counters the cache keeps, which are back at zero after every launch, so
 * two steps on one cache must not overlap in time); otherwise pass 1 and
 * pass 2 are separate launches.  seq_ids: HOST array of n > 0 distinct open
 * sequences; q, k_new, v_new, o_x, lse_x, o, lse, ws: DEVICE pointers laid out
 * as for wsk_append and wsk_attend_gpu; ws of at least
 * wsk_decode_step_workspace() bytes, queried before the call (it does not
 * depend on the new rows).  All checks happen before the routing, so a
 * failed call (other than EHIP) changes nothing.
 * Errors: EINVAL, ESTATE, ERANGE (a full sequence, or L below load_end),
 * ENOMEM, EHIP.
 */
int wsk_decode_step_workspace(const wsk_cache *cache, int32_t n, const int32_t *seq_ids, size_t *bytes);
int wsk_decode_step(wsk_cache *cache, int32_t n, const int32_t *seq_ids, const void *q, const void *k_new,
                    const void *v_new, const float *o_x, const float *lse_x, float *o, float *lse, void *ws,
                    size_t ws_bytes, void *stream);

/*
 * wsk_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same step, with the same arguments minus the workspace.  The chunk
 * partials go to a scratch array that the library keeps in device memory,
 * WSK_NOALLOC_SCRATCH_BYTES per GPU, held from the first wsk_init on that
 * device until the process ends.  The call allocates nothing (no hipMalloc,
 * hipFree or other allocating routine).  Every call on one GPU shares that
 * GPU's array, so calls that overlap on one GPU (different streams, or
 * different host threads) race and must be serialised by the caller; the
 * array keeps the last call's contents, none of which a later call reads
 * before writing it.  Errors: as wsk_decode_step, and ERANGE when the step's
 * chunk partials (wsk_decode_step_workspace) exceed
 * WSK_NOALLOC_SCRATCH_BYTES -- then use wsk_decode_step with a workspace.
 */
#define WSK_NOALLOC_SCRATCH_BYTES (16u << 20)
int wsk_decode_step_noalloc(wsk_cache *cache, int32_t n, const int32_t *seq_ids, const void *q, const void *k_new,
                            const void *v_new, const float *o_x, const float *lse_x, float *o, float *lse,
                            void *stream);

/*
 * One MLA decode step with the output-side expansion folded in (Sec. 6.1:
 * the latent output is expanded by W_UV per head, a linear map that commutes
 * with the LSE merge): wsk_decode_step on an MLA cache, then
 * O[i][h] = W_UV[h]^T O_lat[i][h] (as wsk_mla_expand) in the same workgroups
 * that merge O_lat, which saves the expansion's own launch.  The new rows
 * are k_new (bf16 [n][576], latent | rope); there is no v_new.  o_lat (fp32
 * [n][H][512], 16-byte aligned) receives the merged latent output and may
 * be NULL when only O is wanted; lse as for wsk_decode_step (natural log, in
 * the latent attention's scale); w_uv: DEVICE bf16 [H][512][dv], 16-byte
 * aligned; o: DEVICE fp32 [n][H][dv]; dv one of 64, 128, 256.  q, o_x,
 * lse_x, ws and the workspace size (wsk_decode_step_workspace) as for
 * wsk_decode_step; the caller owns every buffer.  All checks happen before
 * the routing, so a failed call (other than EHIP) changes nothing.
 * Errors: EINVAL (a GQA cache, an unsupported dv, NULL or misaligned
 * pointers, as for wsk_decode_step), ESTATE, ERANGE, ENOMEM, EHIP.
 */
int wsk_decode_step_mla(wsk_cache *cache, int32_t n, const int32_t *seq_ids, const void *q, const void *k_new,
                        const float *o_x, const float *lse_x, const uint16_t *w_uv, int32_t dv, float *o_lat,
                        float *lse, float *o, void *ws, size_t ws_bytes, void *stream);

/*
 * D-window eviction ("flush", Sec. 4.2 and 4.3): for each listed sequence
 * whose D-window [w, L) holds a whole batch, move the batch [w, w') to
 * part[i] (WSK_PART_CPU or WSK_PART_LOAD) and set w = w', where
 * w' = floor((w + D) / block_tokens) * block_tokens (= w + D once w is
 * block-aligned); a sequence with L < w' is left as it is.  moved[i]
 * (optional, HOST) receives w' - w or 0.  The batch's blocks take slots in
 * the destination lowest free first, sequences in ascending id (whatever
 * order seq_ids lists them in), blocks ascending -- the order wsk_append
 * uses; a block that already has a slot there (the CPU slot of the block
 * holding s) keeps it.  The batch's GPU-pool slots are
 * freed.  A kernel on stream gathers the batch's slots, scattered in HBM,
 * in destination order and stores them straight into pinned host memory
 * over the link (where that memory is mapped for the device at its host
 * address; else into the cache's device staging buffer, followed by
 * device -> host DMAs).  To the load region they travel unchanged (the
 * layouts match), one kernel per run of consecutive load slots, into the
 * pinned slots.  To the CPU the kernel rewrites them into the CPU pool's
 * token-major rows, in ~2 MB pieces into a pinned bounce (pinned once, at
 * wsk_init, for caches with evict_tokens > 0), and the host copies each
 * piece's rows into their slots as soon as it lands; the call returns when
 * they are in place.  The part chosen per batch is
 * the caller's: wsk_policy_route_batch gives the paper's roofline routing.
 * Later writes that reuse the freed slots must be ordered after this call on
 * stream.  seq_ids (distinct, open), part, moved: HOST arrays.  Needs
 * evict_tokens > 0 and a device; LOAD needs a load region.
 * All-or-nothing for slot allocation (ENOMEM changes nothing).
 * Errors: EINVAL, ESTATE, ENOMEM, EHIP.
 */
int wsk_flush(wsk_cache *cache, int32_t n, const int32_t *seq_ids, const int32_t *part, int32_t *moved,
              void *stream);

/* The homes of an open sequence's positions [0, L), in order, as runs of one
 * home each (adjacent runs differ): run k is [start[k], end[k]) in part[k]
 * (WSK_PART_*).  count receives the number of runs; at most cap are stored
 * (the arrays may be NULL when cap = 0).  Errors: EINVAL, ESTATE. */
int wsk_seq_segments(const wsk_cache *cache, int32_t seq, int32_t cap, int32_t *start, int32_t *end,
                     int32_t *part, int32_t *count);

/* HOST address of load-region slot `slot` (layout as the GPU pool's slots),
 * for inspection.  The slot's arena must be allocated.  Errors: EINVAL,
 * ERANGE. */
int wsk_load_slot(const wsk_cache *cache, int32_t slot, const void **ptr);

/* Load-region accounting (Sec. 4.3 end): bytes pinned so far, arenas, the
 * seconds spent pinning them, slots in use, and the bytes sent host ->
 * device by wsk_attend_gpu / wsk_attend_blocks and device -> host by
 * wsk_flush since wsk_init. */
typedef struct wsk_load_info {
    int64_t pinned_bytes;
    int64_t slots_used;
    int64_t h2d_bytes;
    int64_t d2h_bytes;
    double pin_seconds;
    int32_t arenas;
    int32_t reserved;
} wsk_load_info;
int wsk_load_stats(const wsk_cache *cache, wsk_load_info *out);

/* ---- roofline split policy (Sec. 5.2, Sec. 5.3) ------------------------- */

/*
 * Per-step latency model of the two engines (Sec. 5.2, Eq. 1):
 *   T_cpu(r) = r A L + c_cpu,   T_gpu(r) = (1 - r) B L + c_gpu
 * A, B: cost per KV token of the CPU and the GPU side (seconds, or any one
 * unit); c_cpu, c_gpu: fixed per-step costs (same unit); r: CPU share of the
 * L placed tokens.  Requires finite values, A, B, c >= 0 and A + B > 0.
 */
typedef struct wsk_roofline {
    double A;
    double B;
    double c_cpu;
    double c_gpu;
} wsk_roofline;

/*
 * The CPU share that balances the two engines at length L >= 1 (Sec. 5.3,
 * Eq. 2): r = clamp(B/(A+B) + (c_gpu - c_cpu)/((A+B) L), 0, 1).  It is the
 * share a sequence of length L is opened with (s = floor(r L),
 * wsk_seq_open).  Errors: EINVAL.
 */
int wsk_roofline_share(const wsk_roofline *model, int64_t L, double *r);

/*
 * Online policy (Sec. 5.3): keeps the model, re-estimates A from the measured
 * CPU latency of recent steps, and routes decode eviction batches so that the
 * running fraction of CPU-placed batches follows the marginal share
 * p = B/(A+B); a sequence opened at share R0 and length L0 then holds
 * R(L) = p + (R0 - p) L0 / L of its tokens on the CPU.
 *   create   model0 with A > 0; window >= 1 steps for the A estimate.
 *   observe  one step's CPU-side latency t_cpu (>= 0, the unit of the model)
 *            and CPU token count n_cpu (>= 0).  A becomes
 *            (sum t - w c_cpu) / sum n over the last w <= window steps; it
 *            is kept when the window has no CPU tokens or the estimate is
 *            not positive.  *A (may be NULL) receives the current A.
 *   route_batch  destination of the next eviction batch: WSK_PART_CPU iff
 *            that leaves the running CPU fraction strictly closer to p (with
 *            c of k batches on the CPU: c + 1/2 < p (k + 1)), else
 *            WSK_PART_GPU.
 *   model    the current model (A estimated; B and the fixed costs as given).
 * A policy is plain host state: not thread-safe, no GPU work.
 * Errors: EINVAL, ENOMEM.
 */
typedef struct wsk_policy wsk_policy;
int wsk_policy_create(const wsk_roofline *model0, int32_t window, wsk_policy **out);
int wsk_policy_destroy(wsk_policy *policy);
int wsk_policy_observe(wsk_policy *policy, double t_cpu, int64_t n_cpu, double *A);
int wsk_policy_route_batch(wsk_policy *policy, int32_t *part);
int wsk_policy_model(const wsk_policy *policy, wsk_roofline *model);

/*
 * Measurement aid, not part of the decode path: reads `bytes` of DEVICE
 * memory at p once with the loads the attention kernels use (16 bytes per
 * lane, 1 KB per wavefront instruction, non-temporal, 32 KB tiles per
 * wavefront), with `workgroups` workgroups of 4 wavefronts taking the tiles
 * in turn (<= 0: 3/4 of the compute units, the count the GQA attention
 * planner aims at), and XORs a 32-bit fold of the data into *out (DEVICE).
 * Timing it gives the plain HBM read rate the attention kernels can be
 * compared with.  p 16-byte aligned; bytes a multiple of 32768.
 * Errors: EINVAL, EHIP.
 */
int wsk_stream_read(const void *p, size_t bytes, int32_t workgroups, uint32_t *out, void *stream);

/*
 * Measurement aid, not part of the decode path: reads `bytes` of HOST memory
 * at p once on `threads` threads of the CPU engine's pool (<= 0: every
 * hardware thread), 64-byte vector loads in 4 MiB pieces, and stores the XOR
 * of its 64-bit words in *out (HOST).  Timing it gives the plain host read
 * rate the CPU engine (wsk_cpu_attend) can be compared with.  bytes a
 * multiple of 8.  Synchronous.  Errors: EINVAL.
 */
int wsk_host_read(const void *p, size_t bytes, int32_t threads, uint64_t *out);

#ifdef __cplusplus
}
#endif

#endif /* WSK_H */
