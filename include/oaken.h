/*
 * oaken.h -- C ABI of the MI355X (gfx950) Oaken KV-cache library.
 *
 * Oaken (Kim et al., ISCA 2025) quantizes each new key/value vector online
 * against four thresholds profiled offline, splitting it into an outer, a middle
 * and an inner group (Sec. 4.3, Eq. 1), shifting outer and middle values by the
 * threshold on their side (Sec. 4.4, Eq. 4), and min-max quantizing each group
 * with a scale computed from that vector alone (Eq. 2-3).  Middle values become
 * 4-bit codes in a dense nibble matrix; inner and outer values are 5-bit codes
 * whose low 4 bits reuse their dense slot and whose remaining information is one
 * 8-bit COO entry (Sec. 4.5).  Decode attention streams the packed pages and
 * dequantizes them on the fly (Sec. 5.2).
 *
 * Conventions for every entry point:
 *   - Data pointers are DEVICE pointers unless stated otherwise; `stream` is a
 *     hipStream_t passed as void* (NULL = default stream).  Work is enqueued
 *     asynchronously on `stream`; the call returns before it completes.
 *   - The caller allocates and owns every buffer (pool, tables, inputs, outputs,
 *     workspace).  The library allocates no device memory and keeps no pointer
 *     after it returns.  Calls on distinct streams are thread-safe.
 *   - Scalars and host pointers are validated before anything is launched; a
 *     failed check returns a non-zero oaken_status and launches nothing.
 *     Device-resident values (lengths, block ids, positions, threshold order)
 *     are preconditions: the library does not read them on the host, and
 *     violating them is undefined behaviour.
 *   - No C++ exception crosses this interface.
 *
 * Quantizer rule (bit-exact contract).  For a vector x[0..d) of finite fp16 values
 * and fp32 thresholds lo_o <= lo_i <= hi_i <= hi_o, in IEEE fp32 with one rounding
 * per operation (no fused multiply-add):
 *   group  OUTER if x < lo_o or x > hi_o; else MIDDLE if x < lo_i or x > hi_i;
 *          else INNER                                                  (Eq. 1)
 *   side   OUTER: x > hi_o; MIDDLE: x > hi_i; INNER: x >= 0
 *   a      OUTER: |x - (side ? hi_o : lo_o)|; MIDDLE: |x - (side ? hi_i : lo_i)|;
 *          INNER: |x|                                                  (Eq. 4)
 *   per group g with b = 3 (MIDDLE) or 4 (INNER, OUTER), L = 2^b - 1:
 *          Min, Max over the group's a (0, 0 if the group is empty);
 *          R = Max - Min; sigma = (R == 0) ? 0 : L / R                 (Eq. 2)
 *          c = clamp(rint_half_even((a - Min) * sigma), 0, L)          (Eq. 3)
 *          code u = side ? 2^b + c : 2^b - 1 - c   (side is the top code bit)
 *          meta   = fp16_rne(Min), fp16_rne(R / L)
 *   COO byte of an INNER/OUTER value at index j:
 *          bit 7 = side, bit 6 = (group == OUTER), bits 5..0 = j mod 64.
 *
 * Page record (one per physical block, KV head, and K or V; P = block_size):
 *   counts  offset 0                     uint8 [P][d/64] COO entries per (slot, chunk)
 *   meta    offset align16(P*d/64)       fp16  [P][6]  (Min, R/L) of INNER, MIDDLE, OUTER
 *   dense   offset align16(meta + 12P)   P*d/2 bytes of nibbles (low nibble first):
 *             K record: token-major,   element j of slot t at byte t*(d/2) + j/2
 *             V record: channel-major, element j of slot t at byte j*(P/2) + t/2
 *           each nibble is the low 4 bits of the element's code
 *   sparse  offset dense + P*d/2         COO bytes, slot-major, then 64-value chunk,
 *           then ascending index; slot t starts at the sum of the counts of slots < t;
 *           capacity P*d bytes (every value an outlier never overflows)
 *   stride  align128(sparse + P*d)
 * The record of (block b, KV head h, which w: 0 = K, 1 = V) starts at
 * pool + ((b * n_kv_heads + h) * 2 + w) * record_stride.
 * Tokens are appended in position order (Sec. 5.2, MMU); writing slot t of a page
 * invalidates any later slot of that page.
 *
 * On-demand sparse pages (the dense and sparse management tables of Sec. 5.2: the
 * sparse matrices vary in size, so their pages are taken as needed).  A cache whose
 * sparse_pool is not NULL keeps each record's COO bytes in a separate pool of
 * OAKEN_SPARSE_PAGE_BYTES-byte sparse pages, taken from a free list as a record's COO
 * stream grows:
 *   counts, meta, dense   as above
 *   table   offset dense + P*d/2         int32 [P*d / OAKEN_SPARSE_PAGE_BYTES]: sparse
 *           page holding bytes [256 i, 256 i + 256) of the record's COO stream (the
 *           stream is laid out as in the fixed record); entries i >= ceil(used / 256),
 *           used = sum of the record's counts, are unused
 *   stride  align128(table + 4 * P*d / OAKEN_SPARSE_PAGE_BYTES)
 * oaken_record_bytes_paged gives that stride.  The free list (sparse_free, int32):
 *   [0] number of free pages n, [1] overflow flag, [2 .. 2+n) the free page ids.
 * oaken_quantize_kv pops pages from it (atomically) and writes their ids into the
 * record's table.  When the list runs dry it sets the overflow flag, and that
 * record's missing pages are left unwritten: the cache contents are then undefined
 * until the pages are released or the pool is reset (attention still only reads
 * inside the pools).  oaken_sparse_release returns retired blocks' pages.
 */
#ifndef OAKEN_H
#define OAKEN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    OAKEN_OK = 0,
    OAKEN_ERR_INVALID_ARG = 1,   /* null pointer, non-positive size, bad ratio, ... */
    OAKEN_ERR_UNSUPPORTED = 2,   /* block_size != 16, head_dim not in {64, 128} */
    OAKEN_ERR_WORKSPACE = 3,     /* workspace missing or smaller than required */
    OAKEN_ERR_HIP = 4            /* the HIP runtime rejected a launch */
} oaken_status;

#define OAKEN_SPARSE_PAGE_BYTES 256

/* One layer's quantized KV cache: host struct describing device buffers. */
typedef struct oaken_cache {
    int32_t num_blocks;          /* physical pages in the pool */
    int32_t block_size;          /* tokens per page P; must be 16 */
    int32_t n_kv_heads;          /* KV heads H */
    int32_t head_dim;            /* d: 64 or 128 */
    int64_t record_stride;       /* oaken_record_bytes(block_size, head_dim), or
                                    oaken_record_bytes_paged(...) with sparse pages */
    void* pool;                  /* device, num_blocks * n_kv_heads * 2 * record_stride bytes */
    const float* thresholds;     /* device fp32 [n_kv_heads][2 (K, V)][4] = lo_o, lo_i, hi_i, hi_o */
    /* On-demand sparse pages; NULL sparse_pool selects the fixed records. */
    void* sparse_pool;           /* device, sparse_pages * OAKEN_SPARSE_PAGE_BYTES bytes */
    int32_t* sparse_free;        /* device, oaken_sparse_free_list_bytes(sparse_pages) bytes */
    int32_t sparse_pages;        /* pages in sparse_pool (>= 1 when sparse_pool is set) */
} oaken_cache;

/* Bytes of one page record (see layout above); -1 if (block_size, head_dim) is unsupported. */
int64_t oaken_record_bytes(int32_t block_size, int32_t head_dim);

/* Bytes of one record with on-demand sparse pages; -1 if unsupported. */
int64_t oaken_record_bytes_paged(int32_t block_size, int32_t head_dim);

/* Bytes of the free list for a pool of sparse_pages pages. */
size_t oaken_sparse_free_list_bytes(int32_t sparse_pages);

/* Marks every sparse page free and clears the overflow flag (run before first use, and
   to drop every sequence at once).  Records keep their bytes: reset them by writing
   their pages again from slot 0.  Enqueued on stream. */
int oaken_sparse_reset(const oaken_cache* cache, void* stream);

/* Retires blocks: their records (every KV head, K and V) give their sparse pages back
   to the free list and become empty (counts zeroed).  block_ids: device int32
   [n_blocks], each < num_blocks, no repeats.  Must not run concurrently with a
   quantize call on the same cache (order them on one stream).  Enqueued on stream. */
int oaken_sparse_release(const oaken_cache* cache, const int32_t* block_ids, int32_t n_blocks,
                         void* stream);

/* Host copies of the free-page count and the overflow flag.  Synchronizes stream. */
int oaken_sparse_status(const oaken_cache* cache, int32_t* free_pages, int32_t* overflowed,
                        void* stream);

/* Host array out[5] = byte offsets of counts, meta, dense, sparse, and the stride.
   Returns OAKEN_OK or OAKEN_ERR_UNSUPPORTED / OAKEN_ERR_INVALID_ARG. */
int oaken_record_layout(int32_t block_size, int32_t head_dim, int64_t* out);

/* Workspace bytes needed by oaken_calibrate_thresholds. */
size_t oaken_calibrate_workspace_bytes(int32_t n_runs, int32_t n_kv_heads);

/* Workspace bytes needed by oaken_decode_attention for these sizes (0 when the
   attention needs none).  The same arguments must be passed to the call. */
size_t oaken_attention_workspace_bytes(int32_t n_seqs, int32_t n_q_heads, int32_t n_kv_heads,
                                       int32_t head_dim, int32_t max_seq_len);

/*
 * Offline threshold profiling (Sec. 4.3 "offline outlier threshold profiling";
 * ratios of Sec. 6.1).  k_calib, v_calib: fp16 [n_runs][tokens_per_run][n_kv_heads]
 * [head_dim].  For each run, head and K|V, with n = tokens_per_run * head_dim values
 *   k_o = rne(n * outer_ratio / 2), k_i = rne(n * inner_ratio)   (computed in fp64)
 *   lo_o = k_o-th smallest value, hi_o = k_o-th largest value (0-based),
 *   t = k_i-th smallest |value| (1-based; 0 if k_i == 0), lo_i = -t, hi_i = t;
 * each threshold is then averaged over runs (fp64 sum in run order, divided by
 * n_runs, rounded once to fp32), the inner pair is clamped into the outer interval
 * (lo_i = min(max(lo_i, lo_o), hi_o), hi_i = max(min(hi_i, hi_o), lo_i)) and -0 becomes +0.
 * Requires 0 <= outer_ratio < 1, 0 <= inner_ratio <= 1, their sum <= 1, 2*k_o <= n-1.
 * Inputs must be finite.  thresholds_out: fp32 [n_kv_heads][2][4].
 * workspace: oaken_calibrate_workspace_bytes(n_runs, n_kv_heads) bytes.
 */
int oaken_calibrate_thresholds(const void* k_calib, const void* v_calib, int32_t n_runs,
                               int32_t tokens_per_run, int32_t n_kv_heads, int32_t head_dim,
                               float outer_ratio, float inner_ratio, float* thresholds_out,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * Online quantization of new key/value rows into the paged cache (Sec. 4.3 "online
 * KV cache quantization", Sec. 4.4-4.5, Sec. 5.2 quantization engine and MMU).
 * k_new, v_new: fp16 [n_tokens][n_kv_heads][head_dim].  Rows cu_tokens[s] ..
 * cu_tokens[s+1]-1 belong to sequence s and land at positions start_pos[s] + i.
 * block_table: int32 [n_seqs][max_blocks_per_seq] maps logical page pos/P to a
 * physical block.  cu_tokens: int32 [n_seqs+1]; start_pos: int32 [n_seqs].
 * max_new_per_seq bounds cu_tokens[s+1]-cu_tokens[s] (it sizes the launch); a
 * sequence with more rows than that may have some of them left unwritten, and
 * nothing outside its own pages is ever written.
 * Preconditions: every block id < num_blocks; each sequence owns its pages; the
 * positions written are the sequence's next positions.
 */
int oaken_quantize_kv(const oaken_cache* cache, const void* k_new, const void* v_new,
                      const int32_t* block_table, int32_t max_blocks_per_seq,
                      const int32_t* start_pos, const int32_t* cu_tokens, int32_t n_seqs,
                      int32_t n_tokens, int32_t max_new_per_seq, void* stream);

/*
 * Batched decode attention over the quantized cache (Sec. 2.1; dequantization
 * engine of Sec. 5.2).  For sequence s and query head h (KV head g = h / (H_q/H)):
 *   out[s][h] = sum_t softmax_t(softmax_scale * q[s][h] . K^[s][g][t]) V^[s][g][t]
 * over t < seq_lens[s], where K^, V^ are the dequantized cache entries:
 *   value = Min + c * Delta, then INNER: +-value, MIDDLE: hi_i + value | lo_i - value,
 *   OUTER: hi_o + value | lo_o - value (upper | lower side).
 * q: fp16 [n_seqs][n_q_heads][head_dim]; out: fp32 [n_seqs][n_q_heads][head_dim].
 * seq_lens: int32 [n_seqs], each in [1, max_seq_len]; block_table as above.
 * Arithmetic is fp32; results match an fp64 evaluation within 2e-3 + 1e-2 |ref|.
 * workspace: oaken_attention_workspace_bytes(n_seqs, n_q_heads, n_kv_heads,
 * head_dim, max_seq_len) bytes, 16-byte aligned (may be NULL when that is 0); it holds
 * the split partials of long sequences.
 */
int oaken_decode_attention(const oaken_cache* cache, const void* q, int32_t n_q_heads,
                           const int32_t* block_table, int32_t max_blocks_per_seq,
                           const int32_t* seq_lens, int32_t n_seqs, int32_t max_seq_len,
                           float softmax_scale, float* out, void* workspace,
                           size_t workspace_bytes, void* stream);

/*
 * Sliding-window decode attention (the Mistral and Mixtral models of Sec. 6.1 attend
 * over a sliding window).  Same as oaken_decode_attention, except that sequence s
 * attends only over its last sliding_window keys:
 *   t in [max(0, seq_lens[s] - sliding_window), seq_lens[s]).
 * sliding_window = 0 means the whole sequence (oaken_decode_attention itself);
 * negative values are rejected.  Keys outside the window are neither read nor
 * weighted; pages wholly before the window are skipped.  workspace:
 * oaken_attention_workspace_bytes_window(..., sliding_window) bytes, which depends
 * on the window (the split plan covers only the pages a window can span).
 */
size_t oaken_attention_workspace_bytes_window(int32_t n_seqs, int32_t n_q_heads, int32_t n_kv_heads,
                                              int32_t head_dim, int32_t max_seq_len,
                                              int32_t sliding_window);

int oaken_decode_attention_window(const oaken_cache* cache, const void* q, int32_t n_q_heads,
                                  const int32_t* block_table, int32_t max_blocks_per_seq,
                                  const int32_t* seq_lens, int32_t n_seqs, int32_t max_seq_len,
                                  int32_t sliding_window, float softmax_scale, float* out,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * Chunked-prefill attention over the quantized cache (prefill reads the KV cache of the
 * earlier tokens, Sec. 2.1; the sliding window of Sec. 6.1 applies per query).  q: fp16
 * [n_tokens][n_q_heads][head_dim], the queries of new tokens; rows cu_tokens[s] ..
 * cu_tokens[s+1]-1 belong to sequence s and sit at positions start_pos[s] + i (the layout
 * and arrays of oaken_quantize_kv).  The query at position p attends causally over its
 * sequence's keys max(0, p + 1 - W) .. p (W = sliding_window, 0 = no window), which must
 * already be in the cache: quantize the chunk's keys and values first.
 * out: fp32 [n_tokens][n_q_heads][head_dim].  Every p + 1 <= max_seq_len.
 * Rows (query token, query head) are processed in blocks: consecutive tokens of one chunk
 * times the query heads of one KV head, up to 16, 32 or 64 rows (sized to the mean chunk,
 * n_tokens / n_seqs; a longer chunk takes several blocks) contracted in fp32, or, at
 * head_dim 128 when the chunks average more than 64 rows per KV head, up to 128 rows on
 * fp16 matrix cores with every real operand split into high and low fp16 parts (fp32
 * accumulation).  A block reads each page of its keys once.
 * workspace: oaken_prefill_attention_workspace_bytes(...) bytes, 16-byte aligned (never 0
 * for valid sizes: it holds the row-block list, and split partials of long prefixes).
 */
size_t oaken_prefill_attention_workspace_bytes(int32_t n_tokens, int32_t n_q_heads, int32_t n_kv_heads,
                                               int32_t head_dim, int32_t max_seq_len, int32_t sliding_window);

int oaken_prefill_attention(const oaken_cache* cache, const void* q, int32_t n_q_heads,
                            const int32_t* block_table, int32_t max_blocks_per_seq, const int32_t* start_pos,
                            const int32_t* cu_tokens, int32_t n_seqs, int32_t n_tokens, int32_t max_seq_len,
                            int32_t sliding_window, float softmax_scale, float* out, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Decode attention without allocation, for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Same computation and arguments as oaken_decode_attention_window, minus the workspace:
 * the split partials live in a scratch array that the library holds in static device
 * memory on each GPU it runs on (OAKEN_NOALLOC_SCRATCH_BYTES per GPU, kept until the
 * process ends; its address is looked up once per device on the first call there).
 * The call allocates nothing.  Sizes whose partials,
 * oaken_attention_workspace_bytes_window(...), exceed OAKEN_NOALLOC_SCRATCH_BYTES are
 * rejected with OAKEN_ERR_WORKSPACE before anything is launched.  Every call on one GPU
 * shares that GPU's scratch and leaves its partials there: calls that overlap on one GPU
 * (other streams, other host threads) race, and the caller must order them.  Nothing in
 * the scratch needs clearing: a call writes every partial it reads.
 */
#define OAKEN_NOALLOC_SCRATCH_BYTES (32u << 20)

int oaken_decode_attention_noalloc(const oaken_cache* cache, const void* q, int32_t n_q_heads,
                                   const int32_t* block_table, int32_t max_blocks_per_seq,
                                   const int32_t* seq_lens, int32_t n_seqs, int32_t max_seq_len,
                                   int32_t sliding_window, float softmax_scale, float* out, void* stream);

/*
 * Measurement helper: a streaming-read probe, for reading the decode attention's achieved
 * bandwidth against what plain loads reach on the same device.  Reads the first
 * bytes_per_record bytes (a multiple of 16, at most 4096) of each of n_records records
 * spaced record_stride bytes apart (a multiple of 16, >= bytes_per_record) from the
 * 16-byte aligned device buffer base, and XORs every 32-bit word read into *checksum
 * (device uint32, which the caller initialises).  A contiguous buffer is read with
 * record_stride == bytes_per_record.  At most 2^31 - 1 chunks of 16 bytes (32 GiB) per
 * call.  Asynchronous on stream.
 */
int oaken_probe_read(const void* base, int64_t bytes_per_record, int64_t record_stride, int64_t n_records,
                     uint32_t* checksum, void* stream);

/* Static description of a status code. */
const char* oaken_status_string(int status);

/* Detail of the last non-OK return on the calling thread ("" if none). */
const char* oaken_last_error(void);

/* ------------------------------------------------------------------------
 * Group-count variants of the quantizer (Sec. 6.2, the number-of-groups study),
 * for measuring accuracy against effective bits.  They write flat per-vector
 * buffers, not page records; decode attention reads only the three-group records.
 *
 * variant: 0 three groups (the default encoding), 1 two groups (outer and middle;
 * COO entry = sign, a zero pad bit, 6-bit index), 2 four groups (two outer levels,
 * one inner), 3 five groups (two outer, two inner) -- 2 and 3 with 9-bit COO entries
 * stored as little-endian uint16 --, 4 and 5 the four- and five-group layouts with
 * 4-bit outliers (3 magnitude bits; the sign is the nibble's top bit and the COO
 * entry keeps 8 bits).  A COO entry is (sign << (6 + r)) | (outlier group rank << 6) |
 * index within the 64-value chunk, r = 1 for up to two outlier groups and 2 otherwise,
 * without the sign for 4-bit outliers; ranks count the outlier groups from the
 * inside out.
 *
 * Boundaries thr8 [n_kv_heads][8] = lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa,
 * hi_ob (outer levels a and b, b outermost; inner levels a and b, b innermost); a
 * variant ignores the levels it does not have.  Groups from the inside out: the
 * innermost (not shifted), inner a (shifted by the b boundary on its side), middle
 * (shifted by the a inner boundary; not shifted without inner groups), outer a
 * (shifted by oa), outer b (shifted by ob).  Middle magnitudes use 3 bits, outliers
 * 4 (or 3); codes are offset binary with the side on top, as in the three-group
 * quantizer.
 *
 * Per vector (x is fp16 [n][n_kv_heads][head_dim], head_dim 64 or 128): nib [d/2]
 * (element j in byte j/2, even j in the low nibble), coo [d * coo_bytes] (entries in
 * chunk then index order), counts [d/64], meta [2 * groups] fp16 (Min, Delta) per
 * group from the inside out, n_coo (int32).  All device pointers; asynchronous on
 * stream.
 * ------------------------------------------------------------------------ */

/* out[6] = outer levels, inner levels, outlier magnitude bits, COO bits, COO bytes,
 * groups.  Host only. */
int oaken_variant_info(int32_t variant, int32_t* out);

int oaken_variant_quantize(int32_t variant, const void* x, int32_t n, int32_t n_kv_heads, int32_t head_dim,
                           const float* thr8, void* nib, void* coo, void* counts, void* meta, int32_t* n_coo,
                           void* stream);

/* out: fp32 [n][n_kv_heads][head_dim], the boundary on the value's side plus or minus
 * Min + code * Delta of its group. */
int oaken_variant_dequantize(int32_t variant, const void* nib, const void* coo, const void* counts,
                             const void* meta, int32_t n, int32_t n_kv_heads, int32_t head_dim,
                             const float* thr8, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OAKEN_H */
