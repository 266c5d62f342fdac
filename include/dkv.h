/*
 * dkv.h -- C ABI of the Distance-KV inference hot path on MI355X (gfx950).
 *
 * Distance-KV keeps a static binary pattern M[layer][query head][distance bin]
 * (Sec. 3.2).  At inference the pattern is mapped to token positions measured
 * from the end of the context (Sec. 3.4, Eq. (4) and Eq. (5)), query heads that
 * share a KV head are combined by union (last paragraph of Sec. 3.4), the KV
 * cache is pruned and packed once in original token order, new tokens are
 * appended and always kept, and decode attends to the packed cache (Sec. 3.4).
 * This library runs those four steps on one GPU:
 *
 *   dkv_map_pattern   pattern -> per-KV-head keep masks and retained lengths
 *                     (dkv_map_pattern_ragged: contexts of different lengths)
 *   dkv_compact       dense K/V + keep mask -> packed K/V, offsets, lengths
 *                     (dkv_compact_bins: map and pack from the pattern in one
 *                     call, whole retained bins copied as blocks;
 *                     dkv_compact_bins_ragged: contexts of different lengths)
 *   dkv_append        new tokens -> free rows after each packed segment
 *   dkv_decode_attn   one decode step of attention over the packed segments
 *   dkv_query_attn    the query block after the context: attention over the
 *                     packed segments plus the block itself, causally
 *   dkv_page_select   zero-copy alternative to the pack: the retained runs
 *                     of a paged cache, listed in place
 *   dkv_paged_decode_attn  decode over a paged cache through those entries
 *   dkv_topk_pattern  the exact-budget export of a pattern from retention
 *                     probabilities (K_rho largest entries)
 *
 * plus dkv_dense_decode_attn, the same attention kernel over an uncompressed
 * cache (the "Dense" comparator of Sec. 4.3).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers are DEVICE pointers unless marked (host).  The caller allocates
 *   and owns every buffer, including workspaces; the library allocates and
 *   frees nothing and keeps no state between calls.
 * - Every call only enqueues work on `stream` (a hipStream_t; NULL is the
 *   default stream) and returns without synchronising.  Buffers must stay
 *   alive until the stream has executed the work.  Calls are re-entrant;
 *   two calls that share an output or a workspace must be ordered by the
 *   caller.
 * - Arguments are checked on the host before anything is enqueued; on any
 *   error nothing is enqueued and the status says why.  DKV_ERR_HIP means the
 *   HIP runtime refused a launch.  Faults inside a kernel surface at the
 *   caller's next synchronisation.
 * - Positions are 0-indexed: position j of a context of length T has
 *   distance delta = T - 1 - j from the last context token.  (Eq. (4) is
 *   written for 1-indexed i = j + 1; with S = 128, R = 1024 and 128-token
 *   bins both give the paper's D = 1013 bins at T = 130,816.)
 * - Query head h belongs to KV head h / G, G = num_q_heads / num_kv_heads.
 * - Element types: DKV_BF16 (K, V, q as bfloat16) or DKV_F32.  Attention
 *   accumulates in fp32 and writes fp32.  head_dim is 64 or 128.  Row and
 *   base pointers of K, V, q, out and packed buffers must be 16-byte aligned.
 * - Sizes: N = num_units (independent (layer, sequence) units),
 *   Hq / Hkv heads, d = head_dim, T = context_len, D = num_bins.
 */
#ifndef DKV_H
#define DKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dkv_status {
  DKV_OK = 0,
  DKV_ERR_INVALID_ARG = 1, /* null pointer, negative or inconsistent size, bad bin edges */
  DKV_ERR_UNSUPPORTED = 2, /* head_dim, group size, bin count or segment count beyond limits */
  DKV_ERR_MISALIGNED = 3,  /* a K/V/q/out/packed pointer is not 16-byte aligned */
  DKV_ERR_CAPACITY = 4,    /* n_tail + n_new exceeds the free rows reserved per segment */
  DKV_ERR_WORKSPACE = 5,   /* workspace missing or smaller than the query function says */
  DKV_ERR_HIP = 6          /* the HIP runtime refused to launch a kernel */
} dkv_status;

typedef enum dkv_dtype { DKV_BF16 = 0, DKV_F32 = 1 } dkv_dtype;

/* Limits (checked; larger values return DKV_ERR_UNSUPPORTED). */
#define DKV_MAX_GROUP 16            /* Hq / Hkv */
#define DKV_MAX_GENERAL_BINS 512    /* bins with arbitrary edges */
#define DKV_MAX_UNIFORM_BINS 16384  /* bins with edges E[k] = W k */
#define DKV_MAX_SEGMENTS 2048       /* batch * num_kv_heads in one decode call */

/*
 * Shape of a pattern-mapping / compaction call (host struct).
 *
 * bin_edges (host) holds D + 1 offsets E[0] = 0 < E[1] < ... < E[D].  A
 * position that is neither sink (j < sink) nor recent (delta < recent) has
 * offset u = delta - recent past the recent window and lies in bin k when
 * E[k] <= u < E[k+1] (Eq. (4); the paper's layout is sink = 128,
 * recent = 1024, E[k] = 128 k).  Positions with u >= E[D] lie in no bin and
 * are pruned: only bins the context covers are instantiated (Sec. 3.4).
 */
typedef struct dkv_layout {
  int32_t num_units;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t context_len;
  int32_t sink;
  int32_t recent;
  int32_t num_bins;
  const int32_t *bin_edges;
} dkv_layout;

/*
 * dkv_map_pattern -- Eq. (5) of Sec. 3.4, then the GQA union.
 *
 * pattern  uint8 [N][Hq][D]; nonzero = bin retained for that query head.
 * kv_mask  out, uint8 [N][Hkv][T]; 1 where any query head of the group keeps
 *          the position (sink and recent positions are always 1), else 0.
 * kv_len   out, int32 [N][Hkv]; number of ones in each kv_mask row.
 * q_mask   out, optional (NULL to skip), uint8 [N][Hq][T]: the per-query-head
 *          logical decision m[l,h,j] of Eq. (5).
 * Limits: D <= DKV_MAX_GENERAL_BINS, or D <= DKV_MAX_UNIFORM_BINS when the
 * edges are uniform.  kv_mask and q_mask must be 16-byte aligned; with
 * context_len = 0 they are not written and may be NULL.
 */
dkv_status dkv_map_pattern(const dkv_layout *layout, const uint8_t *pattern,
                           uint8_t *kv_mask, int32_t *kv_len, uint8_t *q_mask,
                           void *stream);

/*
 * dkv_map_pattern_ragged -- dkv_map_pattern for a batch of contexts of
 * different lengths (e.g. sequences of a serving batch).
 *
 * unit_len  int32 [N] (device): unit n's context is the first unit_len[n]
 *           positions of its mask row (values are clamped to
 *           [0, context_len]).  Eq. (4) and Eq. (5) are applied with that
 *           length: distances count from the end of the unit's own context,
 *           so its sink, recent window and bins move with it, and positions
 *           at or past unit_len[n] are not retained.
 * layout->context_len is the row length of kv_mask, q_mask and the dense
 * cache handed to dkv_compact (the longest context).  Everything else as
 * dkv_map_pattern; packing, append and decode need no change, since they
 * follow the masks and lengths.
 */
dkv_status dkv_map_pattern_ragged(const dkv_layout *layout, const int32_t *unit_len,
                                  const uint8_t *pattern, uint8_t *kv_mask, int32_t *kv_len,
                                  uint8_t *q_mask, void *stream);

/* Workspace bytes dkv_compact needs for this layout (host, no GPU call). */
size_t dkv_compact_workspace_bytes(const dkv_layout *layout);

/*
 * dkv_compact -- the one-time prune and pack of Sec. 3.4 / Fig. 2(b).
 *
 * k, v       dense cache, [N][Hkv][T][d] rows of d elements of `dtype`.
 * kv_mask    uint8 [N][Hkv][T] (nonzero = retained), e.g. from dkv_map_pattern.
 * append_cap free rows reserved after every segment for dkv_append (>= 0).
 * k_out, v_out  packed output, out_rows rows of d elements.  Segment
 *            s = n * Hkv + g starts at seg_off[s] and holds its retained rows
 *            in original token order, followed by append_cap free rows that
 *            this call does not touch.
 * out_rows   capacity of k_out / v_out in rows.  The layout needs
 *            sum_s (kv_len[s] + append_cap) rows.  A segment whose retained
 *            rows and append room would not lie wholly below out_rows is not
 *            packed: nothing of it is written, its seg_len is set to -1 and
 *            its seg_off is clamped to out_rows, so no offset points past
 *            the buffer.  Every call that reads seg_len (dkv_append, the
 *            decode calls, dkv_query_attn) treats a negative length as a
 *            segment with no rows and no room: nothing is appended to it and
 *            its attention outputs are zeros.  *rows_needed reports the true
 *            requirement.
 * seg_off    out, int64 [N*Hkv], row offset of each segment (unit-major).
 * seg_len    out, int32 [N*Hkv], retained rows of each segment (-1: not
 *            packed, see out_rows).
 * src_pos    out, optional int32 [out_rows]: original position j of every
 *            packed row (free rows untouched).
 * rows_needed out, optional int64 [1]: sum_s (seg_len[s] + append_cap).
 * workspace  at least dkv_compact_workspace_bytes(layout) bytes (about
 *            4 * N * Hkv * T: a position list per segment, plus per-tile
 *            counts), no initial contents required.
 * DKV_ERR_UNSUPPORTED when N * Hkv > 65535 or T > 268,435,424 (the copy
 * dispatch, a K and a V workgroup of 256 work-items per 32 packed rows of a
 * segment's T, must hold fewer than 2^32 work-items).
 * The dense cache may be freed once the stream has executed this call: that
 * is what realises the memory reduction.
 */
dkv_status dkv_compact(const dkv_layout *layout, dkv_dtype dtype, const void *k,
                       const void *v, const uint8_t *kv_mask, int32_t append_cap,
                       void *k_out, void *v_out, int64_t out_rows, int64_t *seg_off,
                       int32_t *seg_len, int32_t *src_pos, int64_t *rows_needed,
                       void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes dkv_compact_bins needs for this layout (host, no GPU call);
 * 0 for a layout it does not accept. */
size_t dkv_compact_bins_workspace_bytes(const dkv_layout *layout);

/*
 * dkv_compact_bins -- map and pack in one call, straight from the pattern, as
 * a block gather.  Under Eq. (4)-(5) and the union of Sec. 3.4 a KV head keeps
 * its sink, its recent window and every bin that some query head of its group
 * keeps, and bin k is the contiguous range of positions
 * [T - recent - min(E[k+1], U), T - recent - E[k]) with U = T - sink - recent
 * the compressible span (empty when E[k] >= U).  The packed segment is those
 * ranges in token order, and each is copied as one block of rows (with the
 * paper's 128-token bins of Appendix A: 128 consecutive rows per kept bin).
 * No keep mask is read or written.
 *
 * pattern   uint8 [N][Hq][D] as for dkv_map_pattern.
 * Every other argument as dkv_compact, whose outputs this call reproduces
 * exactly for dkv_map_pattern's kv_mask of the same layout and pattern:
 * k_out, v_out (the retained rows; free rows untouched), seg_off, seg_len
 * (with the same -1 marker for segments that do not fit below out_rows),
 * src_pos and rows_needed.
 * workspace  at least dkv_compact_bins_workspace_bytes(layout) bytes, no
 *            initial contents required.
 * Limits: those of dkv_map_pattern and dkv_compact, N * Hkv <= 65,535 and
 * N * Hkv * (D + 3) <= 2^27 (the workspace's per-segment block tables);
 * beyond them DKV_ERR_UNSUPPORTED.  Other errors as dkv_compact's.
 */
dkv_status dkv_compact_bins(const dkv_layout *layout, dkv_dtype dtype, const void *k,
                            const void *v, const uint8_t *pattern, int32_t append_cap,
                            void *k_out, void *v_out, int64_t out_rows, int64_t *seg_off,
                            int32_t *seg_len, int32_t *src_pos, int64_t *rows_needed,
                            void *workspace, size_t workspace_bytes, void *stream);

/*
 * dkv_compact_bins_ragged -- dkv_compact_bins for a batch of contexts of
 * different lengths (e.g. sequences of a serving batch).
 *
 * unit_len  int32 [N] (device), as for dkv_map_pattern_ragged: unit n's
 *           context is the first unit_len[n] positions of its dense rows
 *           (values are clamped to [0, context_len]); its sink, recent window
 *           and bins count from the end of that context, and positions at or
 *           past it are not retained.
 * The outputs equal dkv_compact's for dkv_map_pattern_ragged's kv_mask of the
 * same layout, lengths and pattern.  The dense rows keep layout->context_len
 * as their stride.  Everything else, limits and errors included, as
 * dkv_compact_bins; DKV_ERR_INVALID_ARG also for a null unit_len with N > 0.
 */
dkv_status dkv_compact_bins_ragged(const dkv_layout *layout, const int32_t *unit_len,
                                   dkv_dtype dtype, const void *k, const void *v,
                                   const uint8_t *pattern, int32_t append_cap, void *k_out,
                                   void *v_out, int64_t out_rows, int64_t *seg_off,
                                   int32_t *seg_len, int32_t *src_pos, int64_t *rows_needed,
                                   void *workspace, size_t workspace_bytes, void *stream);

/*
 * dkv_append -- appended tokens are retained in full (Sec. 3.4).
 *
 * k_new, v_new  [num_segments][n_new][d]; token t of segment s is written to
 *               packed row seg_off[s] + seg_len[s] + n_tail + t.
 * n_tail        (host) tokens already appended to every segment.
 * append_cap    (host) free rows reserved per segment; n_tail + n_new must not
 *               exceed it (DKV_ERR_CAPACITY otherwise).
 * seg_off, seg_len  as returned by dkv_compact; pass seg_off + first segment
 *               to address a subset (e.g. one layer's B * Hkv segments).
 * K is stored already rotated (RoPE at the token's absolute position is the
 * caller's job); the library never re-rotates.
 */
dkv_status dkv_append(dkv_dtype dtype, int32_t num_segments, int32_t head_dim,
                      const void *k_new, const void *v_new, int32_t n_new, int32_t n_tail,
                      int32_t append_cap, void *k_c, void *v_c, const int64_t *seg_off,
                      const int32_t *seg_len, void *stream);

/* Workspace bytes for dkv_decode_attn / dkv_dense_decode_attn (host, no GPU call). */
size_t dkv_decode_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim);

/*
 * dkv_decode_attn -- one decode step over the packed cache (Sec. 3.4).
 *
 * q        [B][Hq][d] queries of this step.
 * k_c, v_c packed cache (shared base pointers of a whole-stack compaction).
 * seg_off, seg_len  the B * Hkv segments of this call, batch-major
 *          (s = b * Hkv + g); for layer l of a stack compacted with units
 *          l * B + b, pass seg_off + l * B * Hkv and seg_len + l * B * Hkv.
 * n_tail   (host) appended tokens per segment; segment s attends rows
 *          [seg_off[s], seg_off[s] + seg_len[s] + n_tail).
 * Every query head of group g attends to all rows of segment (b, g): the
 * union of its group (Sec. 3.4).  out[b][h][:] = softmax(sm_scale * K q) V
 * over those rows, fp32 [B][Hq][d]; a segment with no rows (or seg_len < 0)
 * gives zeros.
 * sm_scale   any value with sm_scale * log2(e) finite in fp32 (negative and
 *          zero included); others return DKV_ERR_INVALID_ARG.  The same rule
 *          holds for every attention call of this library.
 * rows_hint (host) expected total rows of the call (0 = unknown); it only
 * sizes the split, never the result's correctness.
 * workspace  at least dkv_decode_workspace_bytes(...) bytes of scratch for
 *          the split partial results; no initial contents are required.  One
 *          workspace serves one call at a time (calls on one stream are
 *          ordered, so reusing it across a stream's calls is safe).
 * The call enqueues the split attention kernel and, when a segment is split
 * over several workgroups, a combine kernel.
 */
dkv_status dkv_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                           int32_t num_kv_heads, int32_t head_dim, const void *q,
                           const void *k_c, const void *v_c, const int64_t *seg_off,
                           const int32_t *seg_len, int32_t n_tail, float sm_scale,
                           int64_t rows_hint, float *out, void *workspace,
                           size_t workspace_bytes, void *stream);

/*
 * dkv_append_decode_attn -- dkv_append followed by dkv_decode_attn, in one
 * launch: the decode step of a serving loop (Sec. 3.4: a new token's K/V is
 * appended and retained, then the step attends to the packed context plus
 * every appended token).
 *
 * k_new, v_new  [B * Hkv][n_new][d], written to packed rows
 *               seg_off[s] + seg_len[s] + n_tail + t exactly as dkv_append
 *               does; then every segment attends rows
 *               [seg_off[s], seg_off[s] + seg_len[s] + n_tail + n_new).
 * n_tail + n_new must not exceed append_cap (DKV_ERR_CAPACITY).  The result
 * equals the two separate calls with the same rows_hint, bit for bit.
 */
dkv_status dkv_append_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                  int32_t num_kv_heads, int32_t head_dim, const void *q,
                                  const void *k_new, const void *v_new, int32_t n_new,
                                  int32_t n_tail, int32_t append_cap, void *k_c, void *v_c,
                                  const int64_t *seg_off, const int32_t *seg_len, float sm_scale,
                                  int64_t rows_hint, float *out, void *workspace,
                                  size_t workspace_bytes, void *stream);

/*
 * dkv_append_decode_attn_noalloc -- dkv_append_decode_attn for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): the same arguments without the
 * workspace, the same kernels and the same result bit for bit.
 *
 * The split's scratch is a static array of DKV_NOALLOC_SCRATCH_BYTES that
 * the library keeps on every GPU it runs on until the process ends; the call
 * itself allocates and frees nothing.  Shapes whose workspace
 * (dkv_decode_workspace_bytes) exceeds that size return DKV_ERR_UNSUPPORTED.
 * The first call on a device looks the array's address up (DKV_ERR_HIP if
 * that fails).  Every call on one GPU shares that GPU's array: two calls that
 * may overlap on one GPU (different streams, or different host threads)
 * race and must be ordered by the caller.  The array needs no initial
 * contents and keeps whatever the last call left.
 */
#define DKV_NOALLOC_SCRATCH_BYTES (16u << 20)
dkv_status dkv_append_decode_attn_noalloc(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                          int32_t num_kv_heads, int32_t head_dim, const void *q,
                                          const void *k_new, const void *v_new, int32_t n_new,
                                          int32_t n_tail, int32_t append_cap, void *k_c, void *v_c,
                                          const int64_t *seg_off, const int32_t *seg_len,
                                          float sm_scale, int64_t rows_hint, float *out,
                                          void *stream);

/*
 * dkv_dense_decode_attn -- the same attention over an uncompressed cache
 * k, v [B][Hkv][t_cap][d]; every segment attends rows [0, n_valid),
 * n_valid <= t_cap.  Same workspace rules as dkv_decode_attn.
 */
dkv_status dkv_dense_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                 int32_t num_kv_heads, int32_t head_dim, const void *q,
                                 const void *k, const void *v, int64_t t_cap,
                                 int32_t n_valid, float sm_scale, float *out,
                                 void *workspace, size_t workspace_bytes, void *stream);

/*
 * dkv_dense_append_decode_attn -- dense comparator of dkv_append_decode_attn:
 * writes k_new, v_new ([B * Hkv][n_new][d]) to rows n_valid .. n_valid+n_new-1
 * of every dense segment, then attends rows [0, n_valid + n_new).
 * n_valid + n_new must not exceed t_cap (DKV_ERR_CAPACITY).
 */
dkv_status dkv_dense_append_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                        int32_t num_kv_heads, int32_t head_dim, const void *q,
                                        const void *k_new, const void *v_new, int32_t n_new,
                                        void *k, void *v, int64_t t_cap, int32_t n_valid,
                                        float sm_scale, float *out, void *workspace,
                                        size_t workspace_bytes, void *stream);

/* Workspace bytes for dkv_query_attn with the same shapes and rows_hint (host,
 * no GPU call); 0 when the call needs none (workspace may then be NULL). */
size_t dkv_query_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                 int32_t head_dim, int32_t n_q, int64_t rows_hint);

/*
 * dkv_query_attn -- attention of a block of n_q query tokens over the packed
 * cache (Sec. 3.4: after the one-time compaction the query tokens attend to
 * the compressed context, and their own K/V are appended and kept).
 *
 * q        [B][n_q][Hq][d] bf16, token-major (the layout of a model's
 *          activations).
 * The block's K/V must already be appended (dkv_append with n_new = n_q at
 * the same n_tail): segment s = b * Hkv + g then holds the packed context,
 * n_tail earlier appended tokens and the block, and query token i of
 * sequence b, head h (g = h / G) attends to rows
 * [seg_off[s], seg_off[s] + seg_len[s] + n_tail + i + 1): everything before
 * the block, and the block causally up to itself.
 * out      [B][n_q][Hq][d] fp32, softmax(sm_scale * K q) V over those rows.
 *          q, K, V and sm_scale must be finite: outputs for NaN or infinite
 *          inputs are unspecified (the kernels run without NaN semantics).
 * append_cap  free rows reserved per segment; n_tail + n_q <= append_cap.
 * rows_hint (host) total rows the call attends, sum over segments of
 *          seg_len + n_tail + n_q (0 = unknown); it sizes the split of the key
 *          ranges and must equal the value given to dkv_query_workspace_bytes.
 *          A wrong hint changes the split (and the speed), never the result.
 * workspace  dkv_query_workspace_bytes(...) bytes for the split's plan and
 *          per-range partial results (no initial contents required), or NULL
 *          when that is 0 (keys too few to split).
 * Only DKV_BF16 is supported (DKV_ERR_UNSUPPORTED otherwise); head_dim 64 or
 * 128; DKV_ERR_UNSUPPORTED also when a dispatch would exceed 2^32 work-items
 * (512 per workgroup).  When the keys are split the call enqueues a one-workgroup plan
 * kernel, the attention kernel and a combine kernel; otherwise the attention
 * kernel alone.
 */
dkv_status dkv_query_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                          int32_t num_kv_heads, int32_t head_dim, int32_t n_q, const void *q,
                          int32_t n_tail, int32_t append_cap, const void *k_c, const void *v_c,
                          const int64_t *seg_off, const int32_t *seg_len, float sm_scale,
                          int64_t rows_hint, float *out, void *workspace, size_t workspace_bytes,
                          void *stream);

/*
 * Exact-budget pattern export (Sec. 3.3, Eq. (topk-pattern); Appendix A,
 * exact-budget refinement).  The learned pattern keeps the K_rho entries of
 * the L x H x D tensor of retention probabilities with the largest
 * probability, K_rho = round(rho L H D) for a logical retention ratio rho.
 */

/* K_rho = round(rho * L * H * D), halves rounded up (the paper leaves them
 * open), computed in double (host).  Returns -1 unless 0 <= rho <= 1 and the
 * sizes are non-negative. */
int64_t dkv_budget_entries(double rho, int32_t num_layers, int32_t num_q_heads, int32_t num_bins);

/* Workspace bytes of dkv_topk_pattern (host, no GPU call); 0 for an empty or
 * too large tensor. */
size_t dkv_topk_workspace_bytes(int32_t num_layers, int32_t num_q_heads, int32_t num_bins);

/*
 * dkv_topk_pattern -- TopKMask(P, k): pattern[l][h][d] = 1 for the k largest
 * probs[l][h][d] over the whole tensor, 0 elsewhere.
 *
 * probs    float32 [L][Hq][D], 16-byte aligned (any values; NaN ranks below
 *          every number, -0 equals +0).
 * k        0 <= k <= L * Hq * D (DKV_ERR_INVALID_ARG otherwise), e.g.
 *          dkv_budget_entries(rho, L, Hq, D).
 * pattern  out, uint8 [L][Hq][D], 4-byte aligned, with exactly k ones: the
 *          pattern argument of dkv_map_pattern (one unit per layer).
 * workspace  dkv_topk_workspace_bytes(...) bytes, 4-byte aligned, no initial
 *          contents required (DKV_ERR_WORKSPACE otherwise).
 * Ties at the k-th value go to the lowest flat (layer, head, bin) indices, so
 * the result is unique and deterministic.  L * Hq * D < 2^31.  A radix
 * select of five small launches; nothing is read back to the host.
 */
dkv_status dkv_topk_pattern(int32_t num_layers, int32_t num_q_heads, int32_t num_bins,
                            const float *probs, int64_t k, uint8_t *pattern, void *workspace,
                            size_t workspace_bytes, void *stream);

/*
 * Zero-copy paged variant
 * -----------------------
 * The retained set of a segment is its sink, its recent window and a union
 * of whole distance bins (Eq. (4), Eq. (5) and the union of Sec. 3.4), i.e. a
 * few long runs of consecutive positions.  When the cache is kept in pages of
 * page_rows consecutive positions, those runs can be referenced where they
 * are instead of being packed (dkv_compact): with the paper's 128-token bins
 * (Appendix A) and 128-row pages every retained bin is a whole page.
 *
 * Paged cache: K and V pools [num_pages][page_rows][d]; page_table
 * [nseg][pages_per_seg] (int32) gives the physical page that holds positions
 * [p * page_rows, (p + 1) * page_rows) of segment s (logical page p).
 * page_rows is 32, 64, 128, 256, 512 or 1024.
 *
 * Entry: four int32 (physical page, logical page, lo, hi) naming slots
 * [lo, hi) of one page.  A segment's entries are listed in position order:
 * every maximal run of retained context positions within one page, then
 * the append region [T, T + append_cap) page by page.  Decode attends to the
 * slots of the entries whose positions are below T + (tokens appended).
 */
#define DKV_PAGE_ENTRY_INTS 4

/* Workspace bytes of dkv_page_select (host, no GPU call). */
size_t dkv_page_select_workspace_bytes(int32_t num_segments, int32_t context_len);

/*
 * Upper bound on the entries of one segment for keep masks made by
 * dkv_map_pattern with this layout (host): pages of the context, plus one
 * per bin, the sink and the recent window, plus the append region's pages.
 * Returns -1 for invalid arguments.
 */
int64_t dkv_page_entries_bound(const dkv_layout *layout, int32_t append_cap, int32_t page_rows);

/*
 * dkv_page_select -- the zero-copy alternative to dkv_compact: list the
 * retained rows of every segment in place (Sec. 3.4 keeps retained rows in
 * original order; here they keep their original pages too).
 *
 * kv_mask     uint8 [nseg][T], nonzero = retained (e.g. dkv_map_pattern's
 *             kv_mask with nseg = N * Hkv); 16-byte aligned.
 * page_table  int32 [nseg][pages_per_seg]; pages_per_seg * page_rows must be
 *             >= T + append_cap (DKV_ERR_INVALID_ARG otherwise).
 * entries     out, int32 [nseg][max_entries][4], 16-byte aligned.  Entries
 *             at index >= max_entries are not written.
 * n_entries   out, int32 [nseg]: the segment's entry count, even when it is
 *             larger than max_entries (the caller must then enlarge the
 *             array: decode reads at most max_entries entries and cannot
 *             append to a segment whose append entries are missing).
 * seg_len     out, int32 [nseg]: retained context positions (as kv_len).
 * page_used   out, optional uint8 [nseg][pages_per_seg]: 1 for every page an
 *             entry names; pages marked 0 hold no retained row and no append
 *             slot and may be returned to the pool -- that is where the
 *             memory reduction comes from.
 * workspace   dkv_page_select_workspace_bytes(nseg, T) bytes, no initial
 *             contents required.
 * Nothing is copied: the pools are neither read nor written.
 */
dkv_status dkv_page_select(int32_t num_segments, int32_t context_len, int32_t append_cap,
                           int32_t page_rows, const uint8_t *kv_mask, const int32_t *page_table,
                           int32_t pages_per_seg, int32_t max_entries, int32_t *entries,
                           int32_t *n_entries, int32_t *seg_len, uint8_t *page_used,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * dkv_paged_decode_attn -- one decode step over a paged cache (Sec. 3.4),
 * reading the retained rows in place through dkv_page_select's entries.
 *
 * q           [B][Hq][d]; segment s = b * Hkv + g.
 * k_pages, v_pages  the pools, num_pages pages of page_rows rows of d
 *             elements of `dtype`.
 * entries, n_entries, max_entries  as written by dkv_page_select for these
 *             segments (for a subset of a larger selection, offset entries
 *             by first * max_entries * 4 and n_entries by first).
 * context_len T of the selection; n_tail (host) tokens appended so far,
 *             at positions [T, T + n_tail).
 * Every query head of group g attends to the slots of segment (b, g)'s
 * entries whose positions lie below T + n_tail: the retained context and the
 * appended tokens (the union of Sec. 3.4).  An entry that names a page
 * outside [0, num_pages) or slots outside [0, page_rows) attends nothing.
 * The result is that of dkv_decode_attn over a packed cache of the same rows.
 * rows_hint (host) expected sum over segments of entries * page_rows (0 =
 * unknown); it only sizes the split.  out, workspace: as dkv_decode_attn,
 * with the same workspace size (dkv_decode_workspace_bytes).
 */
dkv_status dkv_paged_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                 int32_t num_kv_heads, int32_t head_dim, const void *q,
                                 const void *k_pages, const void *v_pages, int64_t num_pages,
                                 int32_t page_rows, const int32_t *entries,
                                 const int32_t *n_entries, int32_t max_entries,
                                 int32_t context_len, int32_t n_tail, float sm_scale,
                                 int64_t rows_hint, float *out, void *workspace,
                                 size_t workspace_bytes, void *stream);

/*
 * dkv_paged_append_decode_attn -- the decode step of a serving loop over a
 * paged cache: token t of k_new, v_new ([B * Hkv][n_new][d]) is position
 * T + n_tail + t and is written to its slot of the page its append-region
 * entry names (Sec. 3.4: appended and retained), then the step attends as
 * dkv_paged_decode_attn with n_tail + n_new tokens appended, in one launch.
 * append_cap must be the value given to dkv_page_select, and n_tail + n_new
 * must not exceed it (DKV_ERR_CAPACITY).  A segment whose entry count
 * exceeded max_entries is not appended to.
 */
dkv_status dkv_paged_append_decode_attn(dkv_dtype dtype, int32_t batch, int32_t num_q_heads,
                                        int32_t num_kv_heads, int32_t head_dim, const void *q,
                                        const void *k_new, const void *v_new, int32_t n_new,
                                        int32_t n_tail, int32_t append_cap, void *k_pages,
                                        void *v_pages, int64_t num_pages, int32_t page_rows,
                                        const int32_t *entries, const int32_t *n_entries,
                                        int32_t max_entries, int32_t context_len,
                                        float sm_scale, int64_t rows_hint, float *out,
                                        void *workspace, size_t workspace_bytes, void *stream);

/* Static description of a status code. */
const char *dkv_status_string(dkv_status status);

#ifdef __cplusplus
}
#endif

#endif /* DKV_H */
