/*
 * gkv.h -- C ABI of the MI355X (gfx950) graded KV-cache decode-attention library.
 *
 * Method: Geodesia-KV (arXiv 2608.23599).  One layer's KV cache is cut into
 * blocks of P = 64 tokens per (sequence b, KV head h); every block holds one level
 * of a monotone precision ladder (section 3.2): exact fp16, block-scaled 8/4/2-bit
 * scalar codes with fp16 per-channel scale and zero, 4 fp16 centroids with
 * per-token ids, or one fp16 centroid (the block mean).  Single-query (Q = 1) GQA decode attention reads the graded
 * blocks, dequantizing inside an online-softmax loop (section 3.7); optional
 * exact per-page key boxes rank pages for a sparse read (Compressed-Quest,
 * section 3.5); an optional exact residual keeps the tokens with the largest
 * attention-mass x value-error in fp16 (section 3.4, Eq. rdscore).
 *
 * Conventions for every call
 * --------------------------
 *  - Pointers named *_host are host memory; every other data pointer is DEVICE
 *    memory owned by the caller.  No call allocates or frees memory.
 *  - fp16 values travel as uint16_t bit patterns.
 *  - Device work is enqueued on `stream` (a hipStream_t; NULL = default stream)
 *    and is ordered with the caller's other work on that stream.  A call returns
 *    after enqueueing; its results are valid once the stream reaches that point.
 *  - Arguments are validated on the host BEFORE anything is enqueued: a call that
 *    returns an error has enqueued nothing and changed nothing.
 *  - D (head dimension) must be 128 and P (block tokens) 64.  G = Hq / Hkv query
 *    heads share KV head h = g / G (GQA, section 3.1); 1 <= G <= 16.
 *  - Calls are thread-compatible: concurrent calls must not share a cache.
 */
#ifndef GKV_H
#define GKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gkv_status {
  GKV_OK = 0,
  GKV_E_ARG = -1,          /* null pointer, bad enum, non-positive size        */
  GKV_E_SHAPE = -2,        /* D != 128, G out of range, T / capacity mismatch  */
  GKV_E_NOT_MONOTONE = -3, /* a demotion that is not strictly downwards        */
  GKV_E_WORKSPACE = -4,    /* workspace smaller than gkv_workspace_bytes()     */
  GKV_E_HIP = -5,          /* the HIP runtime reported an error                */
  GKV_E_UNSUPPORTED = -6,  /* valid but not implemented combination            */
  GKV_E_POOL = -7          /* a slab pool has no free slot of a needed level    */
} gkv_status;

/* Ladder levels; the numeric value is the bits of a code (1 = centroid state with
 * 4 centroids, 0 = one-centroid state: the block mean, no per-token code).  The
 * numeric order is the ladder order. */
typedef enum gkv_level {
  GKV_MEAN = 0,
  GKV_CENTROID = 1,
  GKV_INT2 = 2,
  GKV_INT4 = 4,
  GKV_INT8 = 8,
  GKV_EXACT = 16
} gkv_level;

/* GKV_VALUES_PER_TOKEN names a value record of a cache with v_per_token set; it is
 * accepted by gkv_decode_record only. */
typedef enum gkv_tensor { GKV_KEYS = 0, GKV_VALUES = 1, GKV_VALUES_PER_TOKEN = 2 } gkv_tensor;

#define GKV_D 128
#define GKV_P 64
#define GKV_KCENT 4

/*
 * Packed record of one tensor block (64 tokens x 128 channels of K or of V)
 * -------------------------------------------------------------------------
 * The layout is chosen so that one 64-lane wavefront loads, with contiguous 16-byte
 * accesses, exactly the operands of its MFMA instructions.  A block is 4 pages of
 * 16 tokens; inside a page, lane l (0..63) owns a chunk of 32 elements x_n
 * (n = 0..31) with kg = l >> 4, m = l & 15:
 *   keys   : x_n = K[token 16*page + m][channel 32*(n>>3) + 8*kg + (n&7)]
 *   values : x_n = V[token 16*page + 4*kg + (n&3)][channel 16*(n>>2) + m]
 * Chunks are stored page-major then lane-major: chunk(page, l) at
 * (page*64 + l) * chunk_bytes.
 *
 * GKV_EXACT   (16384 B): chunks of 32 fp16 values (64 B).
 * GKV_INT8/4/2 (512 + 1024*b B): scale[128] fp16, zero[128] fp16, then chunks of
 *   32 codes (4*b bytes, little-endian 32-bit words).  scale and zero are stored
 *   in lane order: entry 32*kg + n holds the channel of element n of a lane in
 *   group kg (keys: 32*(n>>3) + 8*kg + (n&7); values: 16*(n>>2) + 4*kg + (n&3)).
 *   Code x_n sits in word n / (32/b) at bit position
 *     int8: 8*(n&3)
 *     int4: {4,20,12,28,0,16,8,24}[n&7]
 *     int2: {8,24,14,30,6,22,12,28,4,20,10,26,0,16,2,18}[n&15]
 *   Decoded value = code * scale + zero, exact in fp64 (section 3.2 packed scalar
 *   quantizers; one group per channel over the block's 64 tokens).
 *   Value records of a cache with v_per_token (one group per token over its 128
 *   channels, the grouping of the section 3.2 text) keep the same size and code
 *   layout, with scale[64] and zero[64] fp16 in token order, then 256 unused bytes
 *   (written as zero): decoded value = code * scale[token] + zero[token].
 * GKV_CENTROID (1040 B): 4 x 128 fp16 centroids, then 64 two-bit ids (16 B; the
 *   id of token t is bits 2t..2t+1).  Key centroids are stored [centroid][channel];
 *   value centroids [channel & 15][channel >> 4][centroid].
 * GKV_MEAN (256 B): 128 fp16 values in channel order (keys and values alike); every
 *   token of the block reads this row.
 *
 * Residual rows (section 3.4) are stored as exact-format pseudo-blocks: row r of
 * (b,h) is "token" r & 63 of pseudo-block r >> 6, whose K record is followed by
 * its V record (32768 B per pseudo-block).
 *
 * Page boxes (section 3.5) are fp16 pairs (kmin, kmax) stored per (b, h) as
 * [page >> 6][channel][page & 63][2]; npage_cap must be a multiple of 64.
 */

/* One layer's graded cache.  All device tables are [B][Hkv][capacity]. */
typedef struct gkv_cache {
  int32_t B, Hkv, Hq, D;     /* D must be 128                                        */
  int64_t T;                 /* tokens present (same for every sequence)             */
  int32_t nblk_cap;          /* block-table capacity per (b,h); >= ceil(T/64)        */
  int8_t *level;             /* device [B][Hkv][nblk_cap] gkv_level of each block     */
  int64_t *koff, *voff;      /* device [B][Hkv][nblk_cap] byte offsets into `arena`  */
  uint8_t *arena;            /* device record storage                                */
  int64_t arena_bytes;       /* size of `arena` (offset validation)                  */
  int8_t *level_host;        /* host mirror of `level` (required; kept in sync by the
                                calls that change levels)                            */
  int32_t page;              /* Quest page tokens (16, 32 or 64); 0 = no boxes       */
  int64_t npage_cap;         /* box capacity per (b,h) in pages (multiple of 64)      */
  uint16_t *boxes;           /* device box storage or NULL                           */
  int32_t nres;              /* exact residual rows per (b,h); 0 = none               */
  int32_t nres_cap;          /* residual capacity per (b,h)                           */
  int32_t *res_idx;          /* device [B][Hkv][nres_cap] token index per row, ascending */
  uint8_t *res_rows;         /* device [B][Hkv][ceil(nres_cap/64)] pseudo-blocks      */
  uint64_t *res_mask;        /* device [B][Hkv][nblk_cap] bit t%64 set = token t is
                                read from the residual instead of its block           */
  int32_t *res_off;          /* device [B][Hkv][nblk_cap + 1]: residual rows of the
                                blocks before each block (written by
                                gkv_rd_residual_select; row of token t of block blk =
                                res_off[blk] + popcount of the block's mask below t)  */
  float *cert;               /* device [B][Hkv][nblk_cap][4] or NULL: per block
                                {kerr, verr, vmax, 0} for the decode-time attention
                                error certificate (section 3.6): kerr = max_t
                                ||k_t - k_hat_t||, verr = max_t ||v_t - v_hat_t||
                                against the exact rows, vmax = max_t ||v_t||; written
                                by gkv_quantize_block (keys: kerr; values: verr,
                                vmax), raised by gkv_demote by the change of the
                                reconstruction (triangle inequality) and kept by
                                gkv_append; fp32 rounded upwards                     */
  int32_t v_per_token;       /* 1: the values' int levels are grouped per token (see
                                the record layout); 0: per channel, like the keys     */
  uint64_t version;          /* stamp of the block tables' state: every call that
                                changes level / koff / voff / res_mask / nres or a
                                sequence's block count (gkv_append only when it opens
                                a block) sets a new process-wide unique value; a caller
                                that writes those tables itself calls
                                gkv_cache_changed.  0 = unknown (dense attention plans
                                are then never reused)                                  */
  int64_t *seq_len;          /* device [B] or NULL: sequences of different lengths (the
                                block manager of a serving batch).  seq_len[b] tokens
                                of sequence b are present (0 <= seq_len[b] <= T, and
                                T is the largest), or -1: a retired sequence, which no
                                call reads and gkv_append skips.  NULL: every sequence
                                has T tokens.  The calls that change lengths keep both
                                copies in step.                                         */
  int64_t *seq_len_host;     /* host mirror of seq_len (both NULL or both set)          */
} gkv_cache;

/* Stamps c->version with a new process-wide unique value: a caller that has written
 * the block tables (level, koff, voff, res_mask) or changed nres or a sequence's block
 * count itself calls this before the next attention call, so that a dense plan kept
 * in a workspace for the old tables is not reused.  The library's own calls stamp the
 * cache themselves. */
void gkv_cache_changed(gkv_cache *c);

/* ---------------------------------------------------------------- host helpers */

const char *gkv_strerror(gkv_status s);

/* Bytes of one tensor-block record at `level` (P = 64, D = 128); 0 for a bad level. */
int64_t gkv_block_bytes(int32_t level);

/* Ladder profiles (section 3.2; fixed age ladders of the workloads):
 *   0 "tiny":   newest 4 blocks exact, next 8 int8, next 12 int4, rest int2;
 *   1 "graded": newest 16 exact; int8 / int4 boundaries at 16 + floor(25R/100) and
 *               16 + floor(60R/100), R = nblk - 16; oldest floor(10*nblk/100) blocks
 *               centroid (the exact window takes precedence); rest int2;
 *   2 "exact":  all exact;
 *   3 "rdv2":   newest 16 exact, every older block one-centroid (the low-rate RD-V2
 *               base of section 3.4, used with an exact residual of about 10.2%).
 * Writes levels for blocks 0..nblk-1 (0 = oldest) of a context of T tokens. */
gkv_status gkv_ladder_levels(int32_t profile, int64_t T, int8_t *levels_host, int32_t nblk);

/* Ladder crossings of a context growing to T_new tokens (section 3.2 monotone
 * demotion): compares the profile's levels at T_new with c->level_host for every
 * existing, complete block of every (b,h) and writes up to max_jobs entries
 * jobs_host[3*i..3*i+2] = (b, h, blk), to_host[i] = new level.  With per-sequence
 * lengths every active sequence grows by T_new - c->T tokens and is compared with the
 * profile at its own new length (retired sequences are skipped).  Returns the number
 * of crossings (>= 0), or a negative gkv_status; GKV_E_NOT_MONOTONE if the profile
 * would raise any block's level. */
int32_t gkv_ladder_crossings(const gkv_cache *c, int32_t profile, int64_t T_new, int32_t *jobs_host,
                             int8_t *to_host, int32_t max_jobs);

/* Slab arena: per-level pools of fixed-size slots inside one device buffer.
 * cap[i] = slots for level {16,8,4,2,1,0}[i].  Offsets are byte offsets into the
 * arena; the pool is host-only bookkeeping (single-threaded). */
typedef struct gkv_pool gkv_pool;
gkv_pool *gkv_pool_create(const int64_t cap_host[6]);
int64_t gkv_pool_bytes(const gkv_pool *p);
int64_t gkv_pool_alloc(gkv_pool *p, int32_t level); /* -1 when the pool is full */
gkv_status gkv_pool_free(gkv_pool *p, int32_t level, int64_t offset);
int64_t gkv_pool_used(const gkv_pool *p, int32_t level);
void gkv_pool_destroy(gkv_pool *p);

/* Rate accounting (section 3.5 rate equations; section 4.4 metrics), from the
 * host level mirror.  pages_host = selected pages [B][Hkv][topk] (-1 padded) for a
 * Compressed-Quest read, or NULL for a dense read.  Outputs are bit counts and
 * the number of values Hkv*2*D times the tokens of every sequence (B*T without
 * per-sequence lengths; retired sequences count nothing). */
typedef struct gkv_rates {
  int64_t resident_bits, read_bits, values;
} gkv_rates;
/* A Compressed-Quest read of a cache with residual rows also reads the rows of the
 * residual tokens in its read set (2 * 128 * 16 + 32 bits each) and the 64-bit
 * override mask of every block it touches; res_idx_host = [B][Hkv][nres_cap] host
 * copy of the residual tokens (required then, ignored otherwise). */
gkv_status gkv_account(const gkv_cache *c, const int32_t *pages_host, int32_t topk, const int32_t *res_idx_host,
                       gkv_rates *out);

/* Decode one record (host copy) to codes / values, for inspection and tests.
 * values_host: [64][128] fp64 reconstruction (token-major); codes_host (optional,
 * int levels): [64][128]; scale_host, zero_host (optional, int levels): [128] fp16
 * in channel order ([64] in token order for tensor GKV_VALUES_PER_TOKEN); ids_host (optional, centroid or mean): [64]; cent_host
 * (optional): [4][128] fp16 for a centroid record, [128] for a mean record. */
gkv_status gkv_decode_record(int32_t level, int32_t tensor, const uint8_t *rec_host, double *values_host,
                             int32_t *codes_host, uint16_t *scale_host, uint16_t *zero_host,
                             int32_t *ids_host, uint16_t *cent_host);

/* fp64 -> fp16 bits with one round-to-nearest-even (the conversion the kernels use). */
uint16_t gkv_f64_to_f16(double x);

/* Workspace bytes needed by gkv_quest_select (op 0), gkv_graded_decode_attn (op 1,
 * topk = 0 for a dense read) and gkv_rd_residual_select (op 2).  The size depends on
 * the cache's capacities (not on T), so one workspace serves a cache as it grows.
 * Workspaces need no initialisation; calls that run concurrently need separate
 * workspaces. */
int64_t gkv_workspace_bytes(const gkv_cache *c, int32_t op, int32_t topk);

/* ---------------------------------------------------------------- device calls */

/* Encode blocks [blk_begin, blk_end) of every (b,h) from exact fp16 source rows at
 * the level each block holds in c->level_host, into c->arena at koff/voff
 * (section 3.2 packed quantizers; section 5.7 packed-format constructor).
 * src: [B][Hkv][T_src][128] fp16 keys (which = GKV_KEYS) or values.  Only an exact
 * block may extend past T_src (missing rows are stored as zero).  Int levels use
 * the per-channel asymmetric quantizer z = f16(min), s = f16((max-min)/(2^b-1)),
 * code = rint((x-z)/s) clamped, in fp64; centroid blocks run 4-means Lloyd in fp64
 * (rows 0,16,32,48 initial, at most 10 rounds, fp16 centroids, ids re-assigned
 * against the stored centroids); mean blocks store the fp16 of the block mean (the
 * same iteration with one centroid; the fp64 token-ascending sum is exact).  With
 * per-sequence lengths, blocks at or past a sequence's end are skipped and only an
 * exact block may extend past its length. */
gkv_status gkv_quantize_block(const gkv_cache *c, int32_t which, const uint16_t *src, int64_t T_src,
                              int32_t blk_begin, int32_t blk_end, void *stream);

/* Monotone demotion (section 3.2): re-encode n blocks, each given as
 * jobs_host[3*i .. 3*i+2] = (b, h, blk), from their current record (exact fp64
 * decode) to to_level_host[i], writing the new K and V records at new_koff_host[i]
 * / new_voff_host[i] and updating the device and host level / offset tables.
 * Every job must lower the level (GKV_E_NOT_MONOTONE otherwise; nothing is
 * enqueued then).  A block its sequence does not fill stays exact (GKV_E_SHAPE).
 * The old slots are free once the stream has passed this call. */
gkv_status gkv_demote(gkv_cache *c, int32_t n, const int32_t *jobs_host, const int8_t *to_level_host,
                      const int64_t *new_koff_host, const int64_t *new_voff_host, void *stream);

/* Exact per-page key boxes (section 3.5): for pages [page_begin, page_end) of every
 * (b,h), per channel min and max of the exact fp16 keys k_src [B][Hkv][T_src][128]
 * (all tokens of each page must be < T_src; with per-sequence lengths, pages past a
 * sequence's last complete page are left as they are). */
gkv_status gkv_page_boxes(const gkv_cache *c, const uint16_t *k_src, int64_t T_src, int64_t page_begin,
                          int64_t page_end, void *stream);

/* Append one token per (b,h) (decode step): k_new, v_new [B][Hkv][128] fp16 are
 * written into the newest block, which must be exact.  When the sequence's length is
 * a multiple of 64 a new exact block is opened for its (b,h) units u at byte offsets
 * new_koff_host[u] / new_voff_host[u] (arrays of B*Hkv <= 128 entries; entries of
 * units that open nothing are ignored; may be NULL when no unit opens a block); its
 * other 63 rows are written as zero.  When the token completes a page and boxes are
 * kept, that page's box is written from the exact keys.  c->T is incremented; with
 * per-sequence lengths every active sequence grows by one token at its own position
 * (its rows of k_new / v_new are used, a retired sequence's are ignored) and T
 * becomes the largest length. */
#define GKV_MAX_APPEND_UNITS 128
gkv_status gkv_append(gkv_cache *c, const uint16_t *k_new, const uint16_t *v_new, const int64_t *new_koff_host,
                      const int64_t *new_voff_host, void *stream);

/* Compressed-Quest page selection (section 3.5): for every (b,h), rank the closed
 * pages 0 .. cur-1 (cur = (T-1)/page is always read, never ranked) by the box upper
 * bound UB_g(p) = sum_d q_gd * (q_gd >= 0 ? kmax_pd : kmin_pd), accumulated in
 * fp32 in channel order (each product of two fp16 values is exact in fp32, so every
 * step rounds once), maximised over the group's query heads; write the first topk
 * pages of the order (score desc, page asc) to pages [B][Hkv][topk] in ascending
 * order, -1 padded.  q: [B][Hq][128] fp16, 4-byte aligned (GKV_E_ARG otherwise). */
gkv_status gkv_quest_select(const uint16_t *q, const gkv_cache *c, int32_t topk, int32_t *pages, void *ws,
                            int64_t ws_bytes, void *stream);

/* Fused dequant + online-softmax GQA decode attention (sections 3.1, 3.7): for every
 * query head g of every sequence b, out[b][g][:] = sum_j softmax_j(q.k_j/sqrt(128)) v_j
 * over the read set -- all tokens < T (pages == NULL) or the selected pages
 * [B][Hkv][topk] (ascending and distinct; an entry below 0 or at or past the current
 * page, such as gkv_quest_select's -1 padding, reads nothing) plus the current page
 * (section 3.5).  Residual rows override their
 * tokens' graded entries in both reads (section 3.4).  q: [B][Hq][128] fp16;
 * out: [B][Hq][128] fp32.  Pages may be 16, 32 or 64 tokens (a selected page reads
 * its tiles of one block).  GKV_E_UNSUPPORTED for more than 32767 visits per (b,h)
 * in a dense read (block capacity plus residual pseudo-blocks) or more than 8192
 * read tiles per (b,h) in a Compressed-Quest read (4096 with residual rows). */
gkv_status gkv_graded_decode_attn(const uint16_t *q, const gkv_cache *c, const int32_t *pages, int32_t topk,
                                  float *out, void *ws, int64_t ws_bytes, void *stream);
/* Plan reuse.  The visit plan of a dense read depends only on the block tables, not
 * on the query, and covers each sequence's blocks whole: the attention masks the
 * tokens of a sequence's last (exact) block past its length at run time, so appends
 * that open no block keep the plan.  A dense call whose cache has a nonzero version
 * leaves a tag of the planned state (version, block count, nres, table addresses,
 * split) in the workspace; the plan kernel of a later dense call with the same
 * workspace and an identical tag exits at once and the attention reuses the plan.
 * The check runs on the device, so a captured graph replays it correctly.
 * Compressed-Quest calls always plan (their pages change with every query) and
 * invalidate the tag. */

/* gkv_graded_decode_attn for callers that cannot allocate or pass a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the workspace is a device array inside the library, gkv_noalloc_scratch_bytes()
 * = 32 MiB per GPU, held by each GPU the library runs on until the process ends.
 * The caller passes inputs and outputs as for gkv_graded_decode_attn.
 * GKV_E_WORKSPACE (before anything is enqueued) when the call needs more than the
 * array, i.e. when gkv_workspace_bytes(c, 1, topk) > 32 MiB (a dense read of
 * B * Hkv = 32 (sequence, KV head) units at 2048 blocks with 2621 residual rows
 * each needs about 17 MB).  Every call on one GPU uses that GPU's one array, which
 * keeps the last call's contents: calls that overlap on one GPU (other streams,
 * other threads) race and must be ordered by the caller.  The call itself allocates
 * nothing; its first call on a device looks the array's address up. */
int64_t gkv_noalloc_scratch_bytes(void);
gkv_status gkv_graded_decode_attn_noalloc(const uint16_t *q, const gkv_cache *c, const int32_t *pages, int32_t topk,
                                          float *out, void *stream);

/* Dense gkv_graded_decode_attn plus the decode-time attention error certificate
 * (section 3.6, Eq. certificate) of every query head: bound[b][g] bounds
 * ||o - o_hat|| between attention over the exact rows and out, as
 *   sum_b a_b verr_b + min(2, M+/M- - M-/M+) * max_b vmax_b,
 *   M+- = sum_b a_b exp(+-eps_b),  eps_b = ||q_g|| kerr_b / sqrt(128),
 * with a_b the block's share of out's attention weights and kerr, verr, vmax the
 * cache's per-block numbers (c->cert, required).  Residual rows count as exact.
 * bound: [B][Hq] fp32.  GKV_E_ARG when c->cert is NULL. */
gkv_status gkv_graded_decode_attn_bound(const uint16_t *q, const gkv_cache *c, float *out, float *bound, void *ws,
                                        int64_t ws_bytes, void *stream);

/* The three stages of gkv_graded_decode_attn, for callers that time or schedule them
 * apart; called in this order on one stream with the same cache, pages, topk and
 * workspace they compute the same result.  gkv_attn_plan writes the per-(b,h) visit
 * plan (block records, read tokens, wavefront split) into ws; gkv_attn_partials runs
 * the attention over the plan and leaves one partial (max, sum, output) per
 * workgroup in ws; gkv_attn_merge combines the partials into out.  Arguments and
 * errors as for gkv_graded_decode_attn. */
gkv_status gkv_attn_plan(const gkv_cache *c, const int32_t *pages, int32_t topk, void *ws, int64_t ws_bytes,
                         void *stream);
gkv_status gkv_attn_partials(const uint16_t *q, const gkv_cache *c, const int32_t *pages, int32_t topk, void *ws,
                             int64_t ws_bytes, void *stream);
gkv_status gkv_attn_merge(const gkv_cache *c, const int32_t *pages, int32_t topk, float *out, void *ws,
                          int64_t ws_bytes, void *stream);

/* Sequence lifecycle of a batch with per-sequence lengths (c->seq_len set; the block
 * manager of the paper's serving plug-in).  gkv_retire_sequence gives every block
 * slot of sequence b (all its KV heads, at the levels of c->level_host) back to
 * pool, using the host offset mirrors koff_host / voff_host [B][Hkv][nblk_cap], and
 * marks the sequence retired (-1; T becomes the largest remaining length); the slots
 * are reusable by later work on `stream`.  gkv_admit_sequence makes a retired slot b
 * an empty sequence (length 0), which appends then fill from its first block.  Both
 * update the device length on `stream`.  GKV_E_ARG without per-sequence lengths, for
 * an inactive b (retire) or an active b (admit). */
gkv_status gkv_retire_sequence(gkv_cache *c, gkv_pool *pool, const int64_t *koff_host, const int64_t *voff_host,
                               int32_t b, void *stream);
gkv_status gkv_admit_sequence(gkv_cache *c, int32_t b, void *stream);

/* Rate-distortion exact residual (section 3.4, Eq. rdscore): score every token
 * s_j = a_j * sum_d (v_jd - v_hat_jd)^2 (fp64, channel order, no fused multiply-add)
 * with v_hat its value at its block's level, keep the first nkeep of the order
 * (score desc, token asc) per (b,h), and store their exact K and V rows, ascending
 * indices and per-block override masks in the cache.  k_src, v_src:
 * [B][Hkv][T][128] fp16, 16-byte aligned (rows are read 16 bytes at a time;
 * GKV_E_ARG otherwise); mass: [B][Hkv][T] fp32.  Sets c->nres = nkeep.
 * GKV_E_UNSUPPORTED with per-sequence lengths (the selection runs at prefill, on a
 * batch of one length). */
gkv_status gkv_rd_residual_select(gkv_cache *c, const uint16_t *k_src, const uint16_t *v_src,
                                  const float *mass, int32_t nkeep, void *ws, int64_t ws_bytes,
                                  void *stream);

/* ---------------------------------------------------------------- multi-layer service */

/* One decode step of cache maintenance for L layers (section 3.2: incremental append
 * and monotone demotion; the block-paged serving manager of the paper's plug-in, run
 * natively): for every layer l, append the token k_new[l], v_new[l] (device
 * [L][B][Hkv][128] fp16) as gkv_append does, then demote every block whose level
 * the ladder profile lowers at T + 1, as gkv_demote does.  New exact blocks and the
 * demotion targets take slots from pools[l]; the demoted blocks' old slots are freed
 * to pools[l] (reusable by later work on the same stream).  koff_host[l] and
 * voff_host[l] are host mirrors [B][Hkv][nblk_cap] of layer l's offset tables, kept
 * in sync here.  The layers must share B, Hkv, T and nblk_cap; each layer's
 * crossings are computed from its own levels (layers may hold different levels, as
 * the section 3.3 allocator lays them out).  Before anything is enqueued, every
 * layer's crossings are checked (GKV_E_NOT_MONOTONE when the profile would raise a
 * level of any layer), every slot is taken and checked against its layer's arena:
 * GKV_E_POOL, GKV_E_ARG (a slot past arena_bytes) or any other argument error leaves
 * every cache, pool and mirror unchanged.  A step that opens no block appends up to
 * 16 layers per launch.  Should the HIP runtime fail part-way, the layers whose
 * appends were enqueued keep them (their T advanced; the demotions of a layer after
 * the failure point are not made) and every slot not yet in use goes back to its
 * pool.  Returns the number of blocks demoted over all layers (>= 0) or a
 * negative gkv_status. */
int32_t gkv_layers_step(gkv_cache *const *caches, gkv_pool *const *pools, int64_t *const *koff_host,
                        int64_t *const *voff_host, int32_t L, int32_t profile, const uint16_t *k_new,
                        const uint16_t *v_new, void *stream);

/* ---------------------------------------------------------------- measurement */

/* Streaming-read probe (measurement only, not part of the method): reads `bytes`
 * (a multiple of 16, src 16-byte aligned) with nsink workgroups, each reading one
 * contiguous share with 16-byte nontemporal loads, and writes one word per workgroup
 * to sink [nsink], so that a timed call gives the HBM read rate a plain kernel
 * reaches on this GPU. */
gkv_status gkv_stream_read_probe(const void *src, int64_t bytes, uint32_t *sink, int32_t nsink, void *stream);

/* ---------------------------------------------------------------- observer and allocation */

/* Workspace bytes of gkv_observe_mass for these shapes, or -1 when they are invalid. */
int64_t gkv_observe_ws_bytes(int32_t B, int32_t Hkv, int32_t Hq, int64_t T, int32_t n_obs);

/* Causal attention-mass observer (section 3.1, Eq. 1-2, GQA aggregation and EMA).
 * For every (b, KV head h) the observed queries are the group's G = Hq/Hkv heads at
 * the last n_obs prompt positions T - n_obs .. T - 1; query i sees keys
 * 0 .. T - n_obs + i.  With w = softmax(q . k / sqrt(128)) over the visible keys,
 *   m_new[blk] = mean over the G * n_obs (query, head) rows of sum_{j in blk} w_j,
 * so the masses of one (b, h) sum to 1, and
 *   mass = (1 - alpha) * mass + alpha * m_new   (0 < alpha <= 1; alpha = 1 writes
 *                                                m_new without reading mass).
 * q_obs: [B][n_obs][Hq][128] fp16; k_src: [B][Hkv][T][128] fp16 exact keys;
 * mass: [B][Hkv][ceil(T/64)] fp32.  Logits are fp32 sums of fp16 products (MFMA);
 * the softmax runs in fp32.  GKV_E_UNSUPPORTED when n_obs * G > 512. */
gkv_status gkv_observe_mass(const uint16_t *q_obs, int32_t n_obs, const uint16_t *k_src, int32_t B, int32_t Hkv,
                            int32_t Hq, int64_t T, float alpha, float *mass, void *ws, int64_t ws_bytes,
                            void *stream);

/* qn[b][h] = the largest ||q|| over the group's observed queries q_obs
 * [B][n_obs][Hq][128] fp16 (fp64: channel-ascending sum of squares, then sqrt);
 * the query norm of the bit-depth formula (section 3.3).  qn: [B][Hkv] fp64. */
gkv_status gkv_query_norms(const uint16_t *q_obs, int32_t n_obs, int32_t B, int32_t Hkv, int32_t Hq, double *qn,
                           void *stream);

/* Closed-form level allocation (section 3.3, Eq. allocation solved per block by
 * the analytic bit depth): for every block of every (b, h),
 *   e_b = max over channels of (max - min) of the block's rows of src
 *         [B][Hkv][T][128] fp16: the exact keys (the reading that matches the ||q||
 *         factor) or the exact values (Fig. 1's value error radius) -- the call
 *         takes the range of whichever tensor is passed,
 *   x   = c * qn[b][h] * e_b * N_b * mass[b][h][blk] / (2 tau)  (fp64, left to right;
 *         N_b = ceil(T/64); this is c ||q|| e_b / (2 eps_t) with eps_t = tau/(N_b m_b)),
 *   b*  = ceil(log2(x + 1)), mapped to a level by `rounding`:
 *         GKV_ROUND_UP: the smallest of {1, 2, 4, 8} that is >= b*, else 16 (the
 *           level whose step meets the tolerance; tested as x <= 2^L - 1);
 *         GKV_ROUND_NEAREST: the level of {1, 2, 4, 8, 16} nearest to b*, ties to
 *           the larger ("thresholded to the nearest available discrete level";
 *           x <= 1, 3, 31, 2047 give 1, 2, 4, 8, larger x 16).
 * The newest `window` blocks and a partial last block are exact.  levels: device
 * [B][Hkv][ceil(T/64)] int8 gkv_level.  c > 0 and tau > 0 (the paper leaves both
 * open); GKV_E_ARG for another rounding. */
#define GKV_ROUND_UP 0
#define GKV_ROUND_NEAREST 1
gkv_status gkv_allocate_levels(const uint16_t *src, const float *mass, const double *qn, int32_t B, int32_t Hkv,
                               int64_t T, double c, double tau, int32_t window, int32_t rounding, int8_t *levels,
                               void *stream);

#ifdef __cplusplus
}
#endif
#endif /* GKV_H */
