// Host side of the C ABI declared in include/oaken.h: argument validation, launch
// planning and error reporting.  Nothing here touches device memory contents.
#include "oaken.h"
#include "oaken_internal.h"
#include "prefill_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

// Split partials of oaken_decode_attention_noalloc: static device memory, one copy per
// GPU.  In host code `scratch` only stands for the symbol: its device address comes from
// hipGetSymbolAddress, once per device, and only that address is passed to kernels.
static __device__ __align__(256) uint8_t scratch[OAKEN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

thread_local char g_err[512] = "";

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return status;
}

int ok() {
    g_err[0] = '\0';
    return OAKEN_OK;
}

bool supported_dim(int32_t d) { return d == 64 || d == 128; }

// Tokens the split plan must cover per sequence: a window of W keys can straddle
// (W - 1) / P + 2 pages.
int32_t attention_span(int32_t max_seq_len, int32_t window) {
    if (window <= 0) return max_seq_len;
    const int64_t pages = (int64_t)(window - 1) / oaken::kPage + 2;
    return (int32_t)std::min<int64_t>(max_seq_len, pages * oaken::kPage);
}

int check_cache(const oaken_cache* c) {
    if (!c) return fail(OAKEN_ERR_INVALID_ARG, "cache is NULL");
    if (c->block_size != oaken::kPage)
        return fail(OAKEN_ERR_UNSUPPORTED, "block_size %d unsupported (only 16)", c->block_size);
    if (!supported_dim(c->head_dim))
        return fail(OAKEN_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", c->head_dim);
    if (c->num_blocks <= 0 || c->n_kv_heads <= 0)
        return fail(OAKEN_ERR_INVALID_ARG, "num_blocks and n_kv_heads must be positive");
    const bool paged = c->sparse_pool != nullptr;
    const int64_t want = paged ? oaken::make_layout_paged(c->block_size, c->head_dim).stride
                               : oaken::make_layout(c->block_size, c->head_dim).stride;
    if (c->record_stride != want)
        return fail(OAKEN_ERR_INVALID_ARG, "record_stride %lld != %lld", (long long)c->record_stride,
                    (long long)want);
    if (!c->pool || !c->thresholds) return fail(OAKEN_ERR_INVALID_ARG, "pool or thresholds is NULL");
    if (paged && (!c->sparse_free || c->sparse_pages <= 0))
        return fail(OAKEN_ERR_INVALID_ARG, "sparse pages need a free list and sparse_pages > 0");
    return OAKEN_OK;
}

oaken::SparseArgs sparse_args(const oaken_cache* c) {
    const oaken::Layout L = oaken::make_layout_paged(c->block_size, c->head_dim);
    oaken::SparseArgs a{};
    a.pool = static_cast<uint8_t*>(c->pool);
    a.stride = L.stride;
    a.table = L.sparse;
    a.num_blocks = c->num_blocks;
    a.H = c->n_kv_heads;
    a.cbytes = (int32_t)L.meta;   // counts occupy [0, meta) (padding included)
    a.tbytes = (int32_t)(4 * ((int64_t)c->block_size * c->head_dim / oaken::kSparsePage));
    a.sfree = c->sparse_free;
    a.spages = c->sparse_pages;
    return a;
}

int hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(OAKEN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Decode attention over n_rows sequences.
int attention_rows(const oaken_cache* cache, const void* q, int32_t n_q_heads, const int32_t* block_table,
                   int32_t max_blocks_per_seq, const int32_t* seq_lens, int32_t n_rows, int32_t max_seq_len,
                   int32_t sliding_window,
                   float softmax_scale, float* out, void* workspace, size_t workspace_bytes, void* stream) {
    int st = check_cache(cache);
    if (st != OAKEN_OK) return st;
    if (!q || !block_table || !out)
        return fail(OAKEN_ERR_INVALID_ARG, "a device array argument is NULL");
    if (n_rows <= 0 || max_seq_len <= 0 || max_blocks_per_seq <= 0 || n_q_heads <= 0)
        return fail(OAKEN_ERR_INVALID_ARG, "sizes must be positive");
    if (n_q_heads % cache->n_kv_heads != 0)
        return fail(OAKEN_ERR_INVALID_ARG, "n_q_heads %d not a multiple of n_kv_heads %d", n_q_heads,
                    cache->n_kv_heads);
    if (n_q_heads / cache->n_kv_heads > 8)
        return fail(OAKEN_ERR_UNSUPPORTED, "more than 8 query heads per KV head");
    if ((int64_t)max_blocks_per_seq * oaken::kPage < max_seq_len)
        return fail(OAKEN_ERR_INVALID_ARG, "block table too narrow for max_seq_len");
    if (!std::isfinite(softmax_scale)) return fail(OAKEN_ERR_INVALID_ARG, "softmax_scale not finite");
    if (sliding_window < 0) return fail(OAKEN_ERR_INVALID_ARG, "sliding_window must be >= 0");
    if (cache->sparse_pool && !oaken::mfma_attention_supported(cache->head_dim, n_q_heads / cache->n_kv_heads))
        return fail(OAKEN_ERR_UNSUPPORTED,
                    "on-demand sparse pages need head_dim 128");
    const size_t need = oaken_attention_workspace_bytes_window(n_rows, n_q_heads, cache->n_kv_heads,
                                                               cache->head_dim, max_seq_len, sliding_window);
    if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(OAKEN_ERR_WORKSPACE, "attention workspace %zu < %zu bytes", workspace_bytes, need);
    if (need > 0 && reinterpret_cast<uintptr_t>(workspace) % 16 != 0)
        return fail(OAKEN_ERR_INVALID_ARG, "attention workspace not 16-byte aligned");
    const oaken::SplitPlan sp = oaken::plan_splits(n_rows, n_q_heads, cache->n_kv_heads, cache->head_dim,
                                                   attention_span(max_seq_len, sliding_window));
    oaken::AttnArgs a{};
    a.pool = static_cast<const uint8_t*>(cache->pool);
    a.thr = cache->thresholds;
    a.q = static_cast<const uint16_t*>(q);
    a.block_table = block_table;
    a.seq_lens = seq_lens;
    a.out = out;
    a.partial = static_cast<float*>(workspace);
    a.stride = cache->record_stride;
    a.num_blocks = cache->num_blocks;
    a.H = cache->n_kv_heads;
    a.Hq = n_q_heads;
    a.max_blocks = max_blocks_per_seq;
    a.n_seqs = n_rows;
    a.max_seq_len = max_seq_len;
    a.pages_per_split = sp.pages_per_split;
    a.n_splits = sp.n_splits;
    a.window = sliding_window;
    a.scale = softmax_scale;
    a.spool = static_cast<const uint8_t*>(cache->sparse_pool);
    a.spages = cache->sparse_pages;
    return hip_status(oaken::launch_attention(a, cache->head_dim, static_cast<hipStream_t>(stream)),
                      "attention launch");
}

size_t round_up_sz(size_t v, size_t a) { return (v + a - 1) / a * a; }

// This device's scratch address (looked up on the device's first call); nullptr on error.
void* scratch_address(int& err_status) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        err_status = fail(OAKEN_ERR_HIP, "no usable current device for the scratch (%s)",
                          e != hipSuccess ? hipGetErrorString(e) : "device index out of range");
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            err_status = fail(OAKEN_ERR_HIP, "scratch symbol lookup: %s", hipGetErrorString(e));
            return nullptr;
        }
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

int64_t oaken_record_bytes(int32_t block_size, int32_t head_dim) {
    if (block_size != oaken::kPage || !supported_dim(head_dim)) return -1;
    return oaken::make_layout(block_size, head_dim).stride;
}

int64_t oaken_record_bytes_paged(int32_t block_size, int32_t head_dim) {
    if (block_size != oaken::kPage || !supported_dim(head_dim)) return -1;
    return oaken::make_layout_paged(block_size, head_dim).stride;
}

size_t oaken_sparse_free_list_bytes(int32_t sparse_pages) {
    if (sparse_pages <= 0) return 0;
    return (size_t)(sparse_pages + 2) * sizeof(int32_t);
}

int oaken_sparse_reset(const oaken_cache* cache, void* stream) {
    int st = check_cache(cache);
    if (st != OAKEN_OK) return st;
    if (!cache->sparse_pool) return fail(OAKEN_ERR_INVALID_ARG, "cache has no sparse pages");
    return hip_status(oaken::launch_sparse_reset(sparse_args(cache), static_cast<hipStream_t>(stream)),
                      "sparse reset launch");
}

int oaken_sparse_release(const oaken_cache* cache, const int32_t* block_ids, int32_t n_blocks, void* stream) {
    int st = check_cache(cache);
    if (st != OAKEN_OK) return st;
    if (!cache->sparse_pool) return fail(OAKEN_ERR_INVALID_ARG, "cache has no sparse pages");
    if (n_blocks < 0 || (n_blocks > 0 && !block_ids))
        return fail(OAKEN_ERR_INVALID_ARG, "block_ids NULL or n_blocks negative");
    if (n_blocks == 0) return ok();
    return hip_status(oaken::launch_sparse_release(sparse_args(cache), block_ids, n_blocks,
                                                   static_cast<hipStream_t>(stream)),
                      "sparse release launch");
}

int oaken_sparse_status(const oaken_cache* cache, int32_t* free_pages, int32_t* overflowed, void* stream) {
    int st = check_cache(cache);
    if (st != OAKEN_OK) return st;
    if (!cache->sparse_pool) return fail(OAKEN_ERR_INVALID_ARG, "cache has no sparse pages");
    if (!free_pages || !overflowed) return fail(OAKEN_ERR_INVALID_ARG, "output pointers are NULL");
    int32_t h[2] = {0, 0};
    const hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(h, cache->sparse_free, sizeof(h), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_status(e, "sparse status copy");
    *free_pages = h[0];
    *overflowed = h[1];
    return ok();
}

int oaken_record_layout(int32_t block_size, int32_t head_dim, int64_t* out) {
    if (!out) return fail(OAKEN_ERR_INVALID_ARG, "out is NULL");
    if (block_size != oaken::kPage || !supported_dim(head_dim))
        return fail(OAKEN_ERR_UNSUPPORTED, "unsupported block_size %d / head_dim %d", block_size,
                    head_dim);
    const oaken::Layout L = oaken::make_layout(block_size, head_dim);
    out[0] = L.counts;
    out[1] = L.meta;
    out[2] = L.dense;
    out[3] = L.sparse;
    out[4] = L.stride;
    return ok();
}

size_t oaken_calibrate_workspace_bytes(int32_t n_runs, int32_t n_kv_heads) {
    if (n_runs <= 0 || n_kv_heads <= 0) return 0;
    return (size_t)n_runs * n_kv_heads * 2 * 3 * sizeof(float);
}

size_t oaken_attention_workspace_bytes(int32_t n_seqs, int32_t n_q_heads, int32_t n_kv_heads,
                                       int32_t head_dim, int32_t max_seq_len) {
    return oaken_attention_workspace_bytes_window(n_seqs, n_q_heads, n_kv_heads, head_dim, max_seq_len, 0);
}

size_t oaken_attention_workspace_bytes_window(int32_t n_seqs, int32_t n_q_heads, int32_t n_kv_heads,
                                              int32_t head_dim, int32_t max_seq_len,
                                              int32_t sliding_window) {
    if (n_seqs <= 0 || n_q_heads <= 0 || n_kv_heads <= 0 || n_q_heads % n_kv_heads != 0 ||
        !supported_dim(head_dim) || max_seq_len <= 0)
        return 0;
    const oaken::SplitPlan sp = oaken::plan_splits(n_seqs, n_q_heads, n_kv_heads, head_dim,
                                                   attention_span(max_seq_len, sliding_window));
    if (sp.n_splits <= 1) return 0;
    return (size_t)n_seqs * n_q_heads * sp.n_splits * (head_dim + 2) * sizeof(float);
}

int oaken_calibrate_thresholds(const void* k_calib, const void* v_calib, int32_t n_runs,
                               int32_t tokens_per_run, int32_t n_kv_heads, int32_t head_dim,
                               float outer_ratio, float inner_ratio, float* thresholds_out,
                               void* workspace, size_t workspace_bytes, void* stream) {
    if (!k_calib || !v_calib || !thresholds_out)
        return fail(OAKEN_ERR_INVALID_ARG, "calibration inputs or output NULL");
    if (n_runs <= 0 || tokens_per_run <= 0 || n_kv_heads <= 0 || head_dim <= 0)
        return fail(OAKEN_ERR_INVALID_ARG, "sizes must be positive");
    if (!(outer_ratio >= 0.0f && outer_ratio < 1.0f && inner_ratio >= 0.0f && inner_ratio <= 1.0f &&
          outer_ratio + inner_ratio <= 1.0f))
        return fail(OAKEN_ERR_INVALID_ARG, "ratios (%g, %g) outside [0,1) x [0,1] or sum > 1",
                    (double)outer_ratio, (double)inner_ratio);
    const int64_t n = (int64_t)tokens_per_run * head_dim;
    const int64_t k_o = (int64_t)std::nearbyint((double)n * (double)outer_ratio / 2.0);
    const int64_t k_i = (int64_t)std::nearbyint((double)n * (double)inner_ratio);
    if (2 * k_o > n - 1 || k_i > n)
        return fail(OAKEN_ERR_INVALID_ARG, "outer ratio leaves no middle values (k_o=%lld, n=%lld)",
                    (long long)k_o, (long long)n);
    const size_t need = oaken_calibrate_workspace_bytes(n_runs, n_kv_heads);
    if (!workspace || workspace_bytes < need)
        return fail(OAKEN_ERR_WORKSPACE, "calibration workspace %zu < %zu bytes", workspace_bytes, need);
    oaken::CalibArgs a{};
    a.k = static_cast<const uint16_t*>(k_calib);
    a.v = static_cast<const uint16_t*>(v_calib);
    a.per_run = static_cast<float*>(workspace);
    a.thr_out = thresholds_out;
    a.n = n;
    a.k_o = k_o;
    a.k_i = k_i;
    a.R = n_runs;
    a.T = tokens_per_run;
    a.H = n_kv_heads;
    a.d = head_dim;
    return hip_status(oaken::launch_calibrate(a, static_cast<hipStream_t>(stream)), "calibrate launch");
}

int oaken_quantize_kv(const oaken_cache* cache, const void* k_new, const void* v_new,
                      const int32_t* block_table, int32_t max_blocks_per_seq,
                      const int32_t* start_pos, const int32_t* cu_tokens, int32_t n_seqs,
                      int32_t n_tokens, int32_t max_new_per_seq, void* stream) {
    int st = check_cache(cache);
    if (st != OAKEN_OK) return st;
    if (!k_new || !v_new || !block_table || !start_pos || !cu_tokens)
        return fail(OAKEN_ERR_INVALID_ARG, "a device array argument is NULL");
    if (n_seqs <= 0 || n_tokens < 0 || max_blocks_per_seq <= 0 || max_new_per_seq < 0)
        return fail(OAKEN_ERR_INVALID_ARG, "n_seqs/max_blocks must be positive, counts non-negative");
    if (n_tokens == 0 || max_new_per_seq == 0) return ok();
    oaken::QuantArgs a{};
    a.pool = static_cast<uint8_t*>(cache->pool);
    a.spool = static_cast<uint8_t*>(cache->sparse_pool);
    a.sfree = cache->sparse_free;
    a.spages = cache->sparse_pages;
    a.thr = cache->thresholds;
    a.k_new = static_cast<const uint16_t*>(k_new);
    a.v_new = static_cast<const uint16_t*>(v_new);
    a.block_table = block_table;
    a.start_pos = start_pos;
    a.cu_tokens = cu_tokens;
    a.stride = cache->record_stride;
    a.num_blocks = cache->num_blocks;
    a.H = cache->n_kv_heads;
    a.max_blocks = max_blocks_per_seq;
    a.n_seqs = n_seqs;
    return hip_status(oaken::launch_quantize(a, cache->head_dim, max_new_per_seq,
                                             static_cast<hipStream_t>(stream)),
                      "quantize launch");
}

int oaken_decode_attention(const oaken_cache* cache, const void* q, int32_t n_q_heads,
                           const int32_t* block_table, int32_t max_blocks_per_seq,
                           const int32_t* seq_lens, int32_t n_seqs, int32_t max_seq_len,
                           float softmax_scale, float* out, void* workspace,
                           size_t workspace_bytes, void* stream) {
    return oaken_decode_attention_window(cache, q, n_q_heads, block_table, max_blocks_per_seq, seq_lens,
                                         n_seqs, max_seq_len, 0, softmax_scale, out, workspace,
                                         workspace_bytes, stream);
}

int oaken_decode_attention_window(const oaken_cache* cache, const void* q, int32_t n_q_heads,
                                  const int32_t* block_table, int32_t max_blocks_per_seq,
                                  const int32_t* seq_lens, int32_t n_seqs, int32_t max_seq_len,
                                  int32_t sliding_window, float softmax_scale, float* out,
                                  void* workspace, size_t workspace_bytes, void* stream) {
    if (!seq_lens) return fail(OAKEN_ERR_INVALID_ARG, "a device array argument is NULL");
    return attention_rows(cache, q, n_q_heads, block_table, max_blocks_per_seq, seq_lens, n_seqs,
                          max_seq_len, sliding_window, softmax_scale, out, workspace, workspace_bytes, stream);
}

int oaken_decode_attention_noalloc(const oaken_cache* cache, const void* q, int32_t n_q_heads,
                                   const int32_t* block_table, int32_t max_blocks_per_seq,
                                   const int32_t* seq_lens, int32_t n_seqs, int32_t max_seq_len,
                                   int32_t sliding_window, float softmax_scale, float* out, void* stream) {
    if (!seq_lens) return fail(OAKEN_ERR_INVALID_ARG, "a device array argument is NULL");
    if (!cache) return fail(OAKEN_ERR_INVALID_ARG, "cache is NULL");
    const size_t need = oaken_attention_workspace_bytes_window(n_seqs, n_q_heads, cache->n_kv_heads, cache->head_dim,
                                                               max_seq_len, sliding_window);
    if (need > (size_t)OAKEN_NOALLOC_SCRATCH_BYTES)
        return fail(OAKEN_ERR_WORKSPACE, "split partials need %zu bytes, more than the %u-byte scratch", need,
                    (unsigned)OAKEN_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    if (need > 0) {
        int st = OAKEN_OK;
        ws = scratch_address(st);
        if (!ws) return st;
    }
    return attention_rows(cache, q, n_q_heads, block_table, max_blocks_per_seq, seq_lens, n_seqs,
                          max_seq_len, sliding_window, softmax_scale, out, ws, need, stream);
}

namespace {
// Prefill workspace: [split partials][row blocks: int2 per query token][row-block count]
struct PrefillWs {
    size_t part, blocks, count, total;
};
PrefillWs prefill_ws(int32_t n_tokens, int32_t n_q_heads, int32_t head_dim, const oaken::PrefillPlan& p) {
    PrefillWs w{};
    w.part = p.n_splits > 1 ? round_up_sz((size_t)n_tokens * n_q_heads * p.n_splits * (head_dim + 2) * sizeof(float), 256)
                            : 0;
    w.blocks = round_up_sz((size_t)n_tokens * 2 * sizeof(int32_t), 256);
    w.count = 256;
    w.total = w.part + w.blocks + w.count;
    return w;
}
}  // namespace

size_t oaken_prefill_attention_workspace_bytes(int32_t n_tokens, int32_t n_q_heads, int32_t n_kv_heads,
                                               int32_t head_dim, int32_t max_seq_len, int32_t sliding_window) {
    if (n_tokens <= 0 || n_q_heads <= 0 || n_kv_heads <= 0 || n_q_heads % n_kv_heads != 0 ||
        n_q_heads / n_kv_heads > 8 || !supported_dim(head_dim) || max_seq_len <= 0 || sliding_window < 0)
        return 0;
    // (the call picks the block width from the chunk lengths: room for either plan)
    // (64-row blocks at most: the fewest blocks, hence the most splits any call can plan)
    const oaken::PrefillPlan p0 = oaken::plan_prefill(n_tokens, n_q_heads, n_kv_heads, max_seq_len, sliding_window, false, 4);
    size_t total = prefill_ws(n_tokens, n_q_heads, head_dim, p0).total;
    if (head_dim == 128) {
        const oaken::PrefillPlan p1 = oaken::plan_prefill(n_tokens, n_q_heads, n_kv_heads, max_seq_len, sliding_window, true, 4);
        total = std::max(total, prefill_ws(n_tokens, n_q_heads, head_dim, p1).total);
    }
    return total;
}

int oaken_prefill_attention(const oaken_cache* cache, const void* q, int32_t n_q_heads,
                            const int32_t* block_table, int32_t max_blocks_per_seq, const int32_t* start_pos,
                            const int32_t* cu_tokens, int32_t n_seqs, int32_t n_tokens, int32_t max_seq_len,
                            int32_t sliding_window, float softmax_scale, float* out, void* workspace,
                            size_t workspace_bytes, void* stream) {
    int st = check_cache(cache);
    if (st != OAKEN_OK) return st;
    if (!q || !block_table || !start_pos || !cu_tokens || !out)
        return fail(OAKEN_ERR_INVALID_ARG, "a device array argument is NULL");
    if (n_seqs <= 0 || n_tokens <= 0 || max_seq_len <= 0 || max_blocks_per_seq <= 0 || n_q_heads <= 0)
        return fail(OAKEN_ERR_INVALID_ARG, "sizes must be positive");
    if (n_q_heads % cache->n_kv_heads != 0)
        return fail(OAKEN_ERR_INVALID_ARG, "n_q_heads %d not a multiple of n_kv_heads %d", n_q_heads,
                    cache->n_kv_heads);
    if (n_q_heads / cache->n_kv_heads > 8) return fail(OAKEN_ERR_UNSUPPORTED, "more than 8 query heads per KV head");
    if ((int64_t)max_blocks_per_seq * oaken::kPage < max_seq_len)
        return fail(OAKEN_ERR_INVALID_ARG, "block table too narrow for max_seq_len");
    if (!std::isfinite(softmax_scale)) return fail(OAKEN_ERR_INVALID_ARG, "softmax_scale not finite");
    if (sliding_window < 0) return fail(OAKEN_ERR_INVALID_ARG, "sliding_window must be >= 0");
    const bool wide = oaken::prefill_wide(n_tokens, n_seqs, n_q_heads, cache->n_kv_heads, cache->head_dim);
    const int32_t rt = oaken::prefill_row_tiles(n_tokens, n_seqs, n_q_heads, cache->n_kv_heads);
    const size_t need = oaken_prefill_attention_workspace_bytes(n_tokens, n_q_heads, cache->n_kv_heads,
                                                                cache->head_dim, max_seq_len, sliding_window);
    oaken::PrefillPlan p = oaken::plan_prefill(n_tokens, n_q_heads, cache->n_kv_heads, max_seq_len, sliding_window,
                                               wide, rt);
    // (smaller blocks never plan more splits than the 64-row plan the query sized for; the
    // check keeps that a guarantee)
    if (prefill_ws(n_tokens, n_q_heads, cache->head_dim, p).total > need)
        p = oaken::plan_prefill(n_tokens, n_q_heads, cache->n_kv_heads, max_seq_len, sliding_window, wide, 4);
    const PrefillWs w = prefill_ws(n_tokens, n_q_heads, cache->head_dim, p);
    if (!workspace || workspace_bytes < need)
        return fail(OAKEN_ERR_WORKSPACE, "prefill attention workspace %zu < %zu bytes", workspace_bytes, need);
    if (reinterpret_cast<uintptr_t>(workspace) % 16 != 0)
        return fail(OAKEN_ERR_INVALID_ARG, "prefill attention workspace not 16-byte aligned");
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    oaken::PrefillArgs a{};
    a.pool = static_cast<const uint8_t*>(cache->pool);
    a.thr = cache->thresholds;
    a.q = static_cast<const uint16_t*>(q);
    a.block_table = block_table;
    a.start_pos = start_pos;
    a.cu_tokens = cu_tokens;
    a.row_blocks = reinterpret_cast<const int2*>(ws + w.part);
    a.n_row_blocks = reinterpret_cast<const int32_t*>(ws + w.part + w.blocks);
    a.out = out;
    a.partial = w.part ? reinterpret_cast<float*>(ws) : nullptr;
    a.stride = cache->record_stride;
    a.num_blocks = cache->num_blocks;
    a.H = cache->n_kv_heads;
    a.Hq = n_q_heads;
    a.max_blocks = max_blocks_per_seq;
    a.n_seqs = n_seqs;
    a.n_tokens = n_tokens;
    a.max_seq_len = max_seq_len;
    a.tokens_per_block = p.tokens_per_block;
    // (every row block holds at least one token; a sequence starts a new block)
    a.max_row_blocks = (int32_t)std::min<int64_t>(n_tokens, (n_tokens + p.tokens_per_block - 1) / p.tokens_per_block +
                                                                (int64_t)n_seqs);
    a.pages_per_split = p.pages_per_split;
    a.n_splits = p.n_splits;
    a.window = sliding_window;
    a.scale = softmax_scale;
    a.spool = static_cast<const uint8_t*>(cache->sparse_pool);
    a.spages = cache->sparse_pages;
    a.wide = p.wide ? 1 : 0;
    a.row_tiles = p.row_tiles;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    int rc = hip_status(oaken::launch_prefill(a, cache->head_dim, reinterpret_cast<int2*>(ws + w.part),
                                              reinterpret_cast<int32_t*>(ws + w.part + w.blocks), s),
                        "prefill attention launch");
    if (rc != OAKEN_OK || p.n_splits == 1) return rc;
    oaken::AttnArgs c{};
    c.out = out;
    c.partial = a.partial;
    c.Hq = n_q_heads;
    c.n_seqs = n_tokens;
    c.n_splits = p.n_splits;
    return hip_status(oaken::launch_combine(c, cache->head_dim, s), "prefill combine launch");
}

int oaken_variant_info(int32_t variant, int32_t* out) {
    if (!out) return fail(OAKEN_ERR_INVALID_ARG, "variant info output NULL");
    const oaken::VariantInfo v = oaken::variant_info(variant);
    if (v.groups == 0) return fail(OAKEN_ERR_INVALID_ARG, "unknown variant %d", (int)variant);
    const int32_t vals[6] = {v.n_out, v.n_in, v.out_bits, v.coo_bits, v.coo_bytes, v.groups};
    for (int i = 0; i < 6; ++i) out[i] = vals[i];
    return OAKEN_OK;
}

namespace {
int variant_args(int32_t variant, int32_t n, int32_t n_kv_heads, int32_t head_dim, const float* thr8,
                 oaken::VariantArgs& a) {
    a = oaken::VariantArgs{};
    a.info = oaken::variant_info(variant);
    if (a.info.groups == 0) return fail(OAKEN_ERR_INVALID_ARG, "unknown variant %d", (int)variant);
    if (n < 0 || n_kv_heads <= 0) return fail(OAKEN_ERR_INVALID_ARG, "sizes must be positive");
    if (head_dim != 64 && head_dim != 128)
        return fail(OAKEN_ERR_UNSUPPORTED, "variant encodings support head_dim 64 and 128, not %d", (int)head_dim);
    if (!thr8) return fail(OAKEN_ERR_INVALID_ARG, "boundaries NULL");
    a.thr8 = thr8;
    a.n = n;
    a.H = n_kv_heads;
    return OAKEN_OK;
}
}  // namespace

int oaken_variant_quantize(int32_t variant, const void* x, int32_t n, int32_t n_kv_heads, int32_t head_dim,
                           const float* thr8, void* nib, void* coo, void* counts, void* meta, int32_t* n_coo,
                           void* stream) {
    oaken::VariantArgs a;
    const int st = variant_args(variant, n, n_kv_heads, head_dim, thr8, a);
    if (st != OAKEN_OK) return st;
    if (n == 0) return OAKEN_OK;
    if (!x || !nib || !coo || !counts || !meta || !n_coo) return fail(OAKEN_ERR_INVALID_ARG, "buffer NULL");
    a.x = static_cast<const uint16_t*>(x);
    a.nib = static_cast<uint8_t*>(nib);
    a.coo = static_cast<uint8_t*>(coo);
    a.counts = static_cast<uint8_t*>(counts);
    a.meta = static_cast<uint16_t*>(meta);
    a.n_coo = n_coo;
    return hip_status(oaken::launch_variant_quantize(a, head_dim, static_cast<hipStream_t>(stream)),
                      "variant quantize launch");
}

int oaken_variant_dequantize(int32_t variant, const void* nib, const void* coo, const void* counts,
                             const void* meta, int32_t n, int32_t n_kv_heads, int32_t head_dim,
                             const float* thr8, float* out, void* stream) {
    oaken::VariantArgs a;
    const int st = variant_args(variant, n, n_kv_heads, head_dim, thr8, a);
    if (st != OAKEN_OK) return st;
    if (n == 0) return OAKEN_OK;
    if (!nib || !coo || !counts || !meta || !out) return fail(OAKEN_ERR_INVALID_ARG, "buffer NULL");
    a.nib = const_cast<uint8_t*>(static_cast<const uint8_t*>(nib));
    a.coo = const_cast<uint8_t*>(static_cast<const uint8_t*>(coo));
    a.counts = const_cast<uint8_t*>(static_cast<const uint8_t*>(counts));
    a.meta = const_cast<uint16_t*>(static_cast<const uint16_t*>(meta));
    a.out = out;
    return hip_status(oaken::launch_variant_dequantize(a, head_dim, static_cast<hipStream_t>(stream)),
                      "variant dequantize launch");
}

int oaken_probe_read(const void* base, int64_t bytes_per_record, int64_t record_stride, int64_t n_records,
                     uint32_t* checksum, void* stream) {
    if (!base || !checksum) return fail(OAKEN_ERR_INVALID_ARG, "probe base or checksum NULL");
    if (bytes_per_record <= 0 || bytes_per_record > 4096 || bytes_per_record % 16 != 0)
        return fail(OAKEN_ERR_INVALID_ARG, "bytes_per_record must be a multiple of 16 in [16, 4096]");
    if (record_stride < bytes_per_record || record_stride % 16 != 0 || n_records <= 0)
        return fail(OAKEN_ERR_INVALID_ARG, "record_stride must be a multiple of 16 >= bytes_per_record, n_records > 0");
    if (reinterpret_cast<uintptr_t>(base) % 16 != 0) return fail(OAKEN_ERR_INVALID_ARG, "probe base not 16-byte aligned");
    oaken::ProbeArgs a{};
    a.base = static_cast<const uint8_t*>(base);
    a.record_stride = record_stride;
    a.n_records = n_records;
    a.chunks = (int32_t)(bytes_per_record / 16);
    a.checksum = checksum;
    if (!oaken::prepare_probe(a)) return fail(OAKEN_ERR_INVALID_ARG, "probe reads 2^31 or more 16-byte chunks");
    return hip_status(oaken::launch_probe_read(a, static_cast<hipStream_t>(stream)), "probe launch");
}

const char* oaken_status_string(int status) {
    switch (status) {
        case OAKEN_OK: return "ok";
        case OAKEN_ERR_INVALID_ARG: return "invalid argument";
        case OAKEN_ERR_UNSUPPORTED: return "unsupported configuration";
        case OAKEN_ERR_WORKSPACE: return "workspace missing or too small";
        case OAKEN_ERR_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

const char* oaken_last_error(void) { return g_err; }

}  // extern "C"
