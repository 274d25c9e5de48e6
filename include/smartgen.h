/*
 * smartgen.h — C ABI of the MI355X (gfx950) selective KV-cache transfer hot
 * path of SmartGen (arXiv 2607.28150):
 *
 *   sg_score        per-token importance of every (layer, KV head) from a window
 *                   of prefill attention                     (Section 4.1)
 *   sg_topk         budgeted exact top-k per (request, layer, KV head)
 *                                                           (Section 2.3)
 *   sg_pack         gather of the selected K/V rows into one transfer buffer
 *                                                           (Sections 4.1, 4.2)
 *   sg_split        mask-based KV index splitting and reordering (Algorithm 1)
 *   sg_fetch        copy of indexed rows into paged destination slots
 *                   (parallel on-demand transfer, Section 4.2; non-GDR mode,
 *                   Section 4.4)
 *   sg_decode_attn  decode attention over a partial KV set addressed through a
 *                   page table (Section 2.1; order invariance, Section 4.2);
 *                   sg_decode_attn_noalloc, the same without a workspace
 *   sg_block_importance, sg_block_budget, sg_pack_blocks
 *                   block-granular proactive selection: eq. 1 block
 *                   importance, eq. 2 block budget, and the push of the chosen
 *                   KV blocks (Section 4.1); the global top-K_r of the blocks
 *                   is sg_topk over one row of L * M importances per request
 *   sg_score_count  selection-frequency importance under the alpha-threshold
 *                   selector (Section 4.1, Section 5.1)
 *   sg_score_topshare  selection-frequency importance when each row picks a
 *                   fixed share of its keys (Section 4.1, Section 5.1)
 *   sg_decode_select  decode-time dynamic selection: alpha rule, capped
 *                   (Section 2.3, Section 5.1)
 *   sg_fetch_keep   on-demand fetch that keeps fetched rows in the decode
 *                   side's store and marks them local (reuse, Section 4.2)
 *   sg_spec_quota, sg_spec_push, sg_spec_commit
 *                   speculative transfer of the remaining KV blocks in
 *                   importance order (Section 4.3)
 *
 * Conventions for every call:
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 *     call is asynchronous on it; nothing is synchronised.
 *   - Pointers are caller-owned.  "device" pointers must be readable/writable by
 *     the GPU: device memory, or pinned host memory allocated with
 *     hipHostMalloc (device-accessible through the same address).  The library
 *     never allocates or frees memory; scratch comes from a caller workspace
 *     sized by the matching *_workspace_size call (sg_decode_attn_noalloc uses
 *     a static device array of the library instead).
 *   - Scalars are checked on the host before anything is enqueued; a failing
 *     check returns a negative sg_status, enqueues nothing, and leaves a
 *     description in sg_last_error() (thread-local).  Device-resident metadata
 *     (offsets, indices, page tables) cannot be checked on the host: kernels
 *     clamp every access to the sizes passed here, so a bad entry never reads
 *     or writes outside the arrays; the documented fallback for each call says
 *     what such an entry produces.
 *   - A unit is one (request b, layer l, KV head h).  q head g belongs to KV
 *     head g / G with G = Hq / Hkv (consecutive grouping).
 *   - Varlen batching: cu_seqlens[B+1] (device int32) are the token offsets of
 *     the requests inside T = sum N_b; cu_k[B+1] (device int32) the offsets of
 *     their selected rows inside K_total = sum k_b.
 *   - Element types: SG_F32 (float) or SG_BF16 (bfloat16 stored as uint16).
 *     Head dimension d must be 64 or 128.  Rows are d elements, contiguous;
 *     row starts must be 16-byte aligned (true for d in {64, 128}).
 */
#ifndef SMARTGEN_H
#define SMARTGEN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SG_F32 = 0,
    SG_BF16 = 1,
    /* range markers: a dtype argument may hold any int (others are rejected
       with SG_EINVAL); they give the enum the range of int in C++ too */
    SG_DTYPE_INT_MIN_ = -2147483647 - 1,
    SG_DTYPE_INT_MAX_ = 2147483647
} sg_dtype;

typedef enum {
    SG_OK = 0,
    SG_EINVAL = -1,        /* an argument is out of its documented range */
    SG_EUNSUPPORTED = -2,  /* a valid but unimplemented combination (e.g. d = 96) */
    SG_EWORKSPACE = -3,    /* workspace or destination smaller than required */
    SG_EHIP = -4,          /* the HIP runtime reported an error on launch */
    SG_EINTERNAL = -5
} sg_status;

int sg_version(void);                    /* major*10000 + minor*100 + patch */
const char *sg_status_str(int status);   /* static string for a status code */
const char *sg_last_error(void);         /* detail of this thread's last failure */

/* ---------------------------------------------------------------- sg_score
 * Importance of every cached token (Section 4.1 defines importance as how often
 * attention-magnitude selection picks an entry; this computes its soft,
 * prefill-time form).  For unit (b, l, h) with prompt length N = N_b and the
 * last W prompt positions p_w = N - W + w as queries:
 *
 *   scores[l][h][cu_seqlens[b] + j] =
 *       sum over q heads g of group h, sum over w < W, of
 *       softmax_j( q_win[b][l][g][w] . K[l][h][j] / sqrt(d) ),  causal (j <= p_w)
 *
 * so each unit's scores add up to G * W.
 *
 *   q_win   device, dtype, [B][L][Hq][W][d]: window queries (rows p_w).
 *   k       device, dtype, rows of d; unit (l, h, b) token j is row
 *           l * k_layer_rows + h * T + cu_seqlens[b] + j.  k_layer_rows is
 *           Hkv * T for a per-layer cache, 0 for one source shared by layers.
 *   lse_in  device float [B][L][Hq][W] or NULL: natural-log log-sum-exp of
 *           each window row's scaled causal logits (what a prefill flash
 *           attention produces).  When given, the row statistics pass is
 *           skipped and these values are trusted.
 *   scores  device float [L][Hkv][T] (output).
 *   max_seqlen  host upper bound of every N_b (sizes the launch).
 *   ws      device workspace of at least sg_score_workspace_size(...) bytes.
 * Requirements: W >= 1, W <= N_b for every request (a request with N_b < W gets
 * all-zero scores), G * W <= 512, Hq % Hkv == 0.
 */
size_t sg_score_workspace_size(int B, int L, int Hq, int Hkv, int d, int W, int max_seqlen);
int sg_score(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, int W,
             const int32_t *cu_seqlens, int64_t T, int max_seqlen,
             const void *q_win, const void *k, int64_t k_layer_rows,
             const float *lse_in, float *scores, void *ws, size_t ws_bytes);

/* ---------------------------------------------------------------- sg_score_count
 * Selection-frequency importance under a threshold selector (Section 4.1
 * defines importance as how often the decode-time selector picks an entry;
 * Section 5.1 runs InfiniGen with alpha = 5, which picks the keys whose logit
 * is within alpha of the row's maximum).  The window rows stand in for decode
 * queries as in sg_score:
 *
 *   z_j = q_w . k_j / sqrt(d) (j <= position of row w),  m_w = max_j z_j
 *   counts[l][h][s0 + j] = number of (q head, window row) pairs with
 *                          z_j >= m_w - alpha
 *
 * an integer in [0, G * W] stored as float (so sg_topk ranks it directly;
 * equal counts go to the lower index).  The decision is taken in fp32 on the
 * raw products: q . k_j >= max_j' q . k_j' - alpha * sqrt(d).
 * Arguments, layout and workspace as sg_score (lse_in does not apply; the
 * workspace is required).  alpha must be finite and >= 0.
 */
int sg_score_count(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, int W,
                   const int32_t *cu_seqlens, int64_t T, int max_seqlen,
                   const void *q_win, const void *k, int64_t k_layer_rows,
                   float alpha, float *counts, void *ws, size_t ws_bytes);

/* ---------------------------------------------------------------- sg_score_topshare
 * Selection-frequency importance under the top-share selector (Section 4.1
 * counts how often the selector picks an entry; Section 5.1 gives the other
 * selector setting as the top 20% of the entries).  The window rows stand in
 * for decode queries as in sg_score.  Row w (position p_w = N - W + w) sees
 * n_w = p_w + 1 keys:
 *
 *   z_j  = q_w . k_j / sqrt(d)  (j <= p_w)
 *   k_w  = floor(n_w * ratio_bp / 10000), clamped to [1, n_w]
 *   t_w  = the k_w-th largest z_j of the row
 *   counts[l][h][s0 + j] = number of (q head, window row) pairs with z_j >= t_w
 *
 * so a row picks its k_w largest logits and every key tied with the k_w-th
 * (the threshold is exact: a radix select over the fp32 logits, finished by
 * ranking the few values left in a row's last bin; the decisions are taken in
 * fp32 on the raw products q . k_j, whose order the positive scale keeps; -0
 * equals +0).  Counts are integers in [0, G * W] stored as float, as in
 * sg_score_count.
 *   ratio_bp  the share in basis points, 1 .. 10000 (2000 = 20%).
 *   ws        device workspace of at least sg_score_topshare_workspace_size
 *             bytes (16-byte aligned): per-row thresholds, histograms and
 *             gathered values; its contents need no initialisation.
 * Arguments and layout as sg_score (lse_in does not apply); max_seqlen must be
 * at least every N_b.  A request with N_b < W gets all-zero counts.
 * Calls that share a workspace must be ordered (same stream, or an event).
 */
size_t sg_score_topshare_workspace_size(int B, int L, int Hq, int Hkv, int d, int W, int max_seqlen);
int sg_score_topshare(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, int W,
                      const int32_t *cu_seqlens, int64_t T, int max_seqlen,
                      const void *q_win, const void *k, int64_t k_layer_rows,
                      int ratio_bp, float *counts, void *ws, size_t ws_bytes);

/* ---------------------------------------------------------------- sg_topk
 * Exact top-k of every unit row (Section 2.3: each head of each request keeps
 * its own top-k entries, the KV index of shape BH x k).  Order: larger score
 * first; equal scores by lower token index; -0 equals +0; NaN ranks below every
 * number.  The k_b = cu_k[b+1] - cu_k[b] chosen token ids (request-local,
 * 0 <= id < N_b) are written in ascending order to
 * idx[l][h][cu_k[b] .. cu_k[b+1]).
 *
 *   scores  device float [L][Hkv][T].
 *   idx     device int32 [L][Hkv][K_total] (output).
 *   max_seqlen  host bound of every N_b; must be <= 81920 (80 layers x 1024
 *               blocks when the rows are block importances).
 * A request with k_b > N_b or k_b < 0 (device metadata) gets idx = -1 in its
 * segment.
 */
int sg_topk(void *stream, int B, int L, int Hkv, const int32_t *cu_seqlens, int64_t T,
            int max_seqlen, const int32_t *cu_k, int64_t K_total,
            const float *scores, int32_t *idx);

/* ---------------------------------------------------------------- sg_pack
 * Gathers the selected K and V rows of every unit into one contiguous transfer
 * buffer (the block push of proactive transfer, Section 4.1; a row of selected
 * entries is BH x k x d, Section 4.2).  Layout of dst, S = L * Hkv * K_total:
 *
 *   [ K rows: S x d x esize | V rows: S x d x esize | idx: S x int32 ]
 *
 * slot s = (l * Hkv + h) * K_total + cu_k[b] + i holds the i-th selected row of
 * unit (b, l, h): source row l * kv_layer_rows + h * T + cu_seqlens[b] + idx[s].
 * The index table is idx verbatim.  An index outside [0, N_b) yields a zero row.
 *
 *   k, v    device, dtype, addressed as for sg_score (same layer stride).
 *   idx     device int32 [L][Hkv][K_total].
 *   dst     device memory or pinned host memory (then the kernel writes over
 *           the host link); 16-byte aligned; dst_bytes >= sg_pack_bytes(...).
 *   max_k   host bound of every k_b (>= 0): it sizes the launch (at most
 *           B * max_k slots per row), any k_b is covered, so a tight bound
 *           gives the best grid.
 *   max_workgroups  0, or a budget of workgroups (64 threads each) for the
 *           launch: the call then takes chunks of rows a grid stride apart, at
 *           least one workgroup per (layer, KV head) row.  A pack that runs
 *           beside compute kernels on another stream (the select region's
 *           request groups) disturbs them less with a budget; alone it is
 *           fastest without one.  < 0 -> SG_EINVAL.
 * The call writes the slots [cu_k[0], cu_k[B]) of each (layer, KV head) row,
 * so a group of requests (cu_seqlens and cu_k pointing into the whole batch's
 * arrays, K_total the whole batch's) fills its part of a shared buffer.  A slot
 * in that range that no request's [cu_k[b], cu_k[b+1]) covers (bad offsets)
 * is left unwritten.
 */
size_t sg_pack_bytes(sg_dtype dt, int L, int Hkv, int d, int64_t K_total);
int sg_pack(void *stream, sg_dtype dt, int B, int L, int Hkv, int d,
            const int32_t *cu_seqlens, int64_t T, const int32_t *cu_k, int64_t K_total,
            int max_k, const void *k, const void *v, int64_t kv_layer_rows, const int32_t *idx,
            void *dst, size_t dst_bytes, int max_workgroups);

/* ---------------------------------------------------------------- sg_split
 * Algorithm 1: KV index splitting and (optional) reordering.  Row r holds
 * kv_index[row_off[r] .. row_off[r+1]); its int8 mask row starts at
 * mask[mask_off[r]] and has mask_len[r] entries (0 pad, 1 local, 2 remote;
 * Section 4.2).  The paper shares one mask value across heads; a per-head
 * mask is the general case and is what mask_off addresses.
 *
 *   (1) m_i = mask[kv_index_i] (an index outside [0, mask_len[r]) or a value
 *       other than 1 and 2 counts as 0);
 *   (4)(5) if reorder: out_index row = kv_index row stably sorted by m
 *       descending (remote entries first, then local, then pads);
 *   (2) local = entries with m == 1, (3) remote = entries with m == 2, both in
 *       row order, written from the start of the row's segment;
 *       n_local[r], n_remote[r] count them; the rest of each segment is -1;
 *       n_kept[r] = n_local[r] + n_remote[r] (the row count of a decode set
 *       assembled from both lanes) when n_kept is not NULL.
 *
 *   row_off device int32 [rows+1]; total = row_off[rows] (host copy).
 *   kv_index, out_index, local, remote: device int32 [total]; out_index may be
 *   NULL when reorder == 0.  mask: device int8 of mask_bytes entries; mask_off:
 *   device int64 [rows]; mask_len: device int32 [rows]; n_local, n_remote:
 *   device int32 [rows]; n_kept: device int32 [rows] or NULL.  A mask entry
 *   outside [0, mask_bytes) counts as 0.
 */
int sg_split(void *stream, int rows, const int32_t *row_off, int64_t total,
             const int32_t *kv_index, const int8_t *mask, int64_t mask_bytes,
             const int64_t *mask_off, const int32_t *mask_len, int reorder, int32_t *out_index,
             int32_t *local, int32_t *remote, int32_t *n_local, int32_t *n_remote, int32_t *n_kept);

/* ---------------------------------------------------------------- sg_fetch
 * Copies indexed K/V rows into paged destination slots: the remote lane of
 * parallel on-demand transfer (Section 4.2) with the source in pinned host
 * memory standing in for the prefill node (non-GDR mode, Section 4.4), and the
 * placement of received rows into the decode-side pool.
 *
 * Row r copies its first n_r entries, n_r = n_valid[r] (or the whole segment
 * row_off[r+1] - row_off[r] when n_valid is NULL).  Entry i reads source row
 * src_row_base[r] + index[row_off[r] + i] (+ i when index is NULL) of k_src /
 * v_src and writes logical row L = dst_start[r] + i of the row's destination,
 * i.e. pool row page_table[r * max_pages + L / page_size] + L % page_size of
 * k_pool / v_pool.  Entries whose source row is outside [0, src_rows), whose
 * page is outside the table or whose pool row is outside [0, pool_rows) are
 * skipped.
 *
 *   k_src, v_src  device or pinned host (device-accessible), dtype rows of d.
 *   row_off device int32 [rows+1], total = row_off[rows] (host copy); index
 *   (device int32 [total]) and n_valid (device int32 [rows]) may be NULL;
 *   src_row_base device int64 [rows]; page_table device int32
 *   [rows][max_pages]; dst_start device int32 [rows].
 */
int sg_fetch(void *stream, sg_dtype dt, int d, int rows, const int32_t *row_off, int64_t total,
             const int32_t *index, const int32_t *n_valid,
             const int64_t *src_row_base, int64_t src_rows,
             const void *k_src, const void *v_src,
             const int32_t *page_table, int page_size, int max_pages, const int32_t *dst_start,
             void *k_pool, void *v_pool, int64_t pool_rows);

/* ---------------------------------------------------------------- sg_fetch_keep
 * On-demand fetch with reuse of fetched entries (Section 4.2; the evaluation
 * of Section 5.3 compares against keeping fetched entries).  The copy of
 * sg_fetch, where every fetched entry is also kept in the decode side's KV
 * store at its own token row and its KV mask entry turns local (1), so that a
 * later sg_split finds it local.
 *
 * Row r, entry i < n_r (n_r as in sg_fetch), token t = index[row_off[r] + i]
 * (index is required):
 *   - an entry whose source row src_row_base[r] + t is outside [0, src_rows)
 *     is skipped entirely;
 *   - pool: as sg_fetch (logical row dst_start[r] + i through the page table)
 *     when page_table is not NULL; with page_table NULL, dst_start, k_pool,
 *     v_pool, page_size, max_pages and pool_rows are ignored;
 *   - keep: row keep_row_base[r] + t of k_keep / v_keep when it lies in
 *     [0, keep_rows); only then, when mask is not NULL, 0 <= t < mask_len[r]
 *     and 0 <= mask_off[r] + t < mask_bytes: mask[mask_off[r] + t] = 1.
 *
 *   keep_row_base device int64 [rows]; k_keep, v_keep device, dtype rows of d;
 *   mask device int8 [mask_bytes] or NULL; mask_off device int64 [rows];
 *   mask_len device int32 [rows].  Store rows, pool rows and the mask become
 *   visible to work ordered after the call (stream order or an event); two
 *   entries that write one pool row leave either row.
 */
int sg_fetch_keep(void *stream, sg_dtype dt, int d, int rows, const int32_t *row_off, int64_t total,
                  const int32_t *index, const int32_t *n_valid,
                  const int64_t *src_row_base, int64_t src_rows,
                  const void *k_src, const void *v_src,
                  const int32_t *page_table, int page_size, int max_pages, const int32_t *dst_start,
                  void *k_pool, void *v_pool, int64_t pool_rows,
                  const int64_t *keep_row_base, void *k_keep, void *v_keep, int64_t keep_rows,
                  int8_t *mask, int64_t mask_bytes, const int64_t *mask_off, const int32_t *mask_len);

/* ---------------------------------------------------------------- sg_decode_attn
 * Decode attention over a partial KV set (Section 2.1; Section 4.2 notes that
 * the order of entries does not change the result).  For sequence b and q head
 * g (KV head h = g / G):
 *
 *   n = min(n_rows[b][h], max_pages * page_size); logical row i lives at pool
 *   row page_table[b][h][i / page_size] + i % page_size;
 *   out[b][g] = sum_i softmax_i(scale * q[b][g] . k_i) * v_i      (fp32)
 *
 * No causal mask (a decode query sees every row of its set).  Rows whose pool
 * index is outside [0, pool_rows) are left out; an empty set gives zeros.
 *
 *   q       device, dtype, [B][Hq][d].
 *   k_pool, v_pool  device, dtype, [pool_rows][d].
 *   page_table device int32 [B][Hkv][max_pages]; n_rows device int32 [B][Hkv].
 *   out     device float [B][Hq][d] (output).
 *   ws      device workspace >= sg_decode_attn_workspace_size(...) bytes.
 * Batching layers of one step is B' = L * B independent sequences.
 * Requirements: 1 <= G <= 16, page_size >= 1.
 */
size_t sg_decode_attn_workspace_size(int B, int Hq, int Hkv, int d, int max_pages, int page_size);
int sg_decode_attn(void *stream, sg_dtype dt, int B, int Hq, int Hkv, int d, float scale,
                   const void *q, const void *k_pool, const void *v_pool, int64_t pool_rows,
                   const int32_t *page_table, const int32_t *n_rows, int page_size, int max_pages,
                   float *out, void *ws, size_t ws_bytes);

/* ---------------------------------------------------------------- sg_decode_attn_noalloc
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * operation, arguments and kernels as sg_decode_attn, without a workspace.
 * The split states live in a static device array of the library (one per
 * GPU, sg_decode_attn_noalloc_scratch_bytes() = 16 MiB, held until the
 * process ends); its device address is resolved once per device on the first
 * call there, with that device current.  The call allocates and frees
 * nothing.  A call whose split states would need more than the array holds
 * returns SG_EWORKSPACE and enqueues nothing (sg_decode_attn with a caller
 * workspace serves it).  Every call on one GPU shares that GPU's array and
 * every split state is written before it is read, so nothing needs clearing;
 * calls that overlap on one GPU (other streams, other threads) race on it and
 * must be ordered by the caller.
 */
size_t sg_decode_attn_noalloc_scratch_bytes(void);
int sg_decode_attn_noalloc(void *stream, sg_dtype dt, int B, int Hq, int Hkv, int d, float scale,
                           const void *q, const void *k_pool, const void *v_pool, int64_t pool_rows,
                           const int32_t *page_table, const int32_t *n_rows, int page_size, int max_pages,
                           float *out);

/* ---------------------------------------------------------------- block mode
 * Block-granular proactive selection (Section 4.1).  Per layer the sequence of
 * a request (N tokens) is cut into M KV blocks of Nb = ceil(N / M) tokens;
 * block m holds tokens [m*Nb, min((m+1)*Nb, N)) in every KV head.
 *
 * sg_block_importance: eq. 1 over measured per-entry scores,
 *   imp[b][l][m] = +inf                                     for l = 0, 1
 *                = mean over the block's (head, token) entries of
 *                  scores[l][h][cu_seqlens[b] + t]         for l >= 2,
 *   and -inf for a block without tokens (trailing blocks when N is not a
 *   multiple of M).  fp32 sums in a fixed order, so results repeat exactly.
 *     scores  device float [L][Hkv][T]; imp device float [B][L][M] (output).
 *
 * sg_block_budget (host only): eq. 2, the number of blocks whose transfer can
 *   overlap the prefill of all but the first layer,
 *     K_r = floor(M (L - 1) Tp / Tt), clipped to [2M, L M]
 *   (Tt = 0 gives L M).  Returns -1 for M < 1, L < 1 or negative times.
 *   The blocks are then chosen with sg_topk over one row per request:
 *   L' = Hkv' = 1, cu_seqlens' = (0, L M, 2 L M, ...), cu_k' = offsets of the
 *   per-request K_r; ids come out ascending as c = l * M + m.
 *
 * sg_pack_blocks: the chosen blocks of one request (tokens [s0, s0 + N) of the
 *   source rows) into one buffer, S = nblk * Hkv * Nb rows per tensor,
 *     [ K rows: S x d x esize | V rows: S x d x esize | ids: nblk x int32 ]
 *   Slot row (s * Hkv + h) * Nb + r holds source row
 *   l * kv_layer_rows + h * T + s0 + m * Nb + r of block ids[s] = l * M + m;
 *   rows past the prompt end, and every row of an id outside [0, L M), are
 *   zero.  k, v: device (or pinned host), rows of d elements, at least
 *   (L - 1) * kv_layer_rows + Hkv * T rows; ids: device int32 [nblk];
 *   dst: device or host-mapped pinned, >= sg_pack_blocks_bytes(...) bytes.
 *   Requires s0 + N <= T and N > 0 when nblk > 0.
 */
int sg_block_importance(void *stream, int B, int L, int Hkv, const int32_t *cu_seqlens, int64_t T, int M,
                        const float *scores, float *imp);
int64_t sg_block_budget(int M, int L, double Tp, double Tt);
size_t sg_pack_blocks_bytes(sg_dtype dt, int Hkv, int d, int64_t N, int M, int nblk);
int sg_pack_blocks(void *stream, sg_dtype dt, int L, int Hkv, int d, int64_t T, int64_t s0, int64_t N, int M,
                   const void *k, const void *v, int64_t kv_layer_rows, int nblk, const int32_t *ids,
                   void *dst, size_t dst_bytes);

/* ---------------------------------------------------------------- sg_decode_select
 * Decode-time dynamic KV selection (Section 2.3: each decode step's selector
 * picks KV entries from the step's query; Section 5.1: InfiniGen's alpha = 5,
 * partial ratio 0.3 and a maximum KV selection ratio of 20%).  For request b,
 * layer l and KV head h, with the G q heads of its group and the request's
 * N = N_b keys:
 *
 *   z[g][j] = scale * q[b][l][g] . K[l][h][j],     m_g = max_j z[g][j]
 *   r_j     = max over g of (z[g][j] - m_g)        (<= 0; 0 at each maximum)
 *   S       = { j : r_j >= -alpha }                (some head of the group picks j)
 *
 * If |S| exceeds cap_b = cu_cap[b+1] - cu_cap[b], the cap_b entries with the
 * largest r_j are kept (ties: lower j).  The kept ids go ascending to
 * idx[l][h][cu_cap[b] ...], n_sel[b][l][h] counts them, and the rest of the
 * segment is -1 (which sg_split drops as a pad).  r and the rule are computed
 * in fp32.
 *
 *   d       row width: the whole head (64, 128) or a partial set of its
 *           channels (32, 40, 48; InfiniGen speculates with 30% of them); q and
 *           k hold the same d channels.
 *   scale   logit scale, 1/sqrt(full head dimension); 0 means 1/sqrt(d).
 *   q       device, dtype, [B][L][Hq][d] (the step's queries).
 *   k       device, dtype, rows of d; unit (b, l, h) token j is row
 *           l * k_layer_rows + h * T + cu_seqlens[b] + j.
 *   cu_cap  device int32 [B+1]; idx device int32 [L][Hkv][K_cap] (output);
 *   n_sel   device int32 [B][L][Hkv] (output).
 *   ws      device workspace of sg_decode_select_workspace_size(...) bytes
 *           (the logits of every q head).
 * Requirements: G in {1, 2, 4, 8}, max_seqlen <= 32768, alpha and scale
 * finite and >= 0.
 */
size_t sg_decode_select_workspace_size(int B, int L, int Hq, int max_seqlen);
int sg_decode_select(void *stream, sg_dtype dt, int B, int L, int Hq, int Hkv, int d, const void *q,
                     const int32_t *cu_seqlens, int64_t T, int max_seqlen, const void *k, int64_t k_layer_rows,
                     float scale, float alpha, const int32_t *cu_cap, int64_t K_cap, int32_t *idx,
                     int32_t *n_sel, void *ws, size_t ws_bytes);

/* ---------------------------------------------------------------- speculative transfer
 * Speculative transfer (Section 4.3): while the decode side computes
 * attention, the prefill side pushes the KV blocks that the proactive transfer
 * left behind, in importance order (eq. 1), a fixed fraction of all blocks
 * (the speculative ratio) per transfer, and updates the KV mask.
 *
 * sg_spec_quota (host only): blocks per transfer, ceil(blocks * ratio_bp /
 *   10000) clipped to [1, blocks] (0 for blocks = 0), so 1 / ratio transfers
 *   deliver every block.  Returns -1 for blocks < 0, ratio_bp < 1 or overflow.
 *
 * The blocks of one transfer are the quota's top entries of `rem`, a float row
 * of the L * M importances of a request in which every delivered block is NaN
 * (sg_topk ranks NaN last): sg_topk(rem, k = min(quota, blocks left)).
 *
 * sg_spec_push: delivers blocks ids[0 .. nblk) of one request (tokens
 *   [s0, s0 + N) of T, blocks of Nb = ceil(N / M) tokens).  For an id
 *   c = l * M + m in [0, L M), every KV head h and block token
 *   t = m * Nb + r < N:
 *     k_dst, v_dst row l * dst_layer_rows + h * T + s0 + t
 *         = k_src, v_src row l * src_layer_rows + h * T + s0 + t
 *     mask[(l * Hkv + h) * T + s0 + t] = 1                 (local)
 *   and rem[c] = NaN when rem is not NULL.  Other ids are skipped.
 *   k_src, v_src: device or pinned host (the prefill side), at least
 *   (L - 1) * src_layer_rows + Hkv * T rows (a stride of 0 shares one source
 *   across layers); k_dst, v_dst: device (the decode side's store), at least
 *   (L - 1) * dst_layer_rows + Hkv * T rows; ids device int32 [nblk]; mask
 *   device int8 [L][Hkv][T] or NULL (rows only: no mask or rem update; see
 *   sg_spec_commit); rem device float [L M] or NULL.  Requires
 *   s0 + N <= T and N > 0 when nblk > 0.  Store rows, mask and rem become
 *   visible to work ordered after the call (stream order or an event).
 */
int64_t sg_spec_quota(int64_t blocks, int ratio_bp);
int sg_spec_push(void *stream, sg_dtype dt, int L, int Hkv, int d, int64_t T, int64_t s0, int64_t N, int M,
                 const void *k_src, const void *v_src, int64_t src_layer_rows, void *k_dst, void *v_dst,
                 int64_t dst_layer_rows, int nblk, const int32_t *ids, int8_t *mask, float *rem);

/* sg_spec_commit: the marking half of sg_spec_push on its own.  For every
 *   delivered block id c = l * M + m in ids[0 .. nblk), every KV head h and
 *   block token t = m * Nb + r < N: mask[(l * Hkv + h) * T + s0 + t] = 1, and
 *   rem[c] = NaN when rem is not NULL; other ids are skipped.
 *   The paper's transfer puts a block's rows before its mask update with
 *   in-order delivery (Section 4.3).  Here a push without a mask
 *   (sg_spec_push with mask = NULL moves the rows only, on a side stream)
 *   lets the decode steps go on; once the push has completed, the consumer
 *   enqueues sg_spec_commit on its own stream, ordered after the push (an
 *   event), so no step reads a local entry whose row has not landed.
 *   ids device int32 [nblk]; mask device int8 [L][Hkv][T]; rem device float
 *   [L M] or NULL.  Requires s0 + N <= T and N > 0 when nblk > 0.
 */
int sg_spec_commit(void *stream, int L, int Hkv, int64_t T, int64_t s0, int64_t N, int M, int nblk,
                   const int32_t *ids, int8_t *mask, float *rem);

#ifdef __cplusplus
}
#endif
#endif /* SMARTGEN_H */
