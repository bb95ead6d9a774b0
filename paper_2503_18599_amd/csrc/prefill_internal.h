// Private declarations of the chunked-prefill attention (attention_prefill.hip, api.hip),
// kept apart from the decode-attention declarations.
#pragma once

#include "oaken_internal.h"

namespace oaken {

// Chunked prefill (attention_prefill.hip): row blocks of (query token, query head) rows of
// one sequence's chunk and one KV head, each reading its pages once.
struct PrefillArgs {
    const uint8_t* pool;
    const float* thr;             // [H][2][4]
    const uint16_t* q;            // fp16 bits [n_tokens][Hq][d]
    const int32_t* block_table;   // [n_seqs][max_blocks]
    const int32_t* start_pos;     // [n_seqs]
    const int32_t* cu_tokens;     // [n_seqs + 1]
    const int2* row_blocks;       // (sequence, first chunk token) per row block
    const int32_t* n_row_blocks;  // number of row blocks (device)
    float* out;                   // fp32 [n_tokens][Hq][d]
    float* partial;               // [n_tokens][Hq][n_splits][d + 2] when n_splits > 1
    int64_t stride;
    int32_t num_blocks, H, Hq, max_blocks, n_seqs, n_tokens, max_seq_len;
    int32_t tokens_per_block, max_row_blocks, pages_per_split, n_splits, window;
    float scale;
    const uint8_t* spool;         // on-demand sparse pages (nullptr: fixed records)
    int32_t spages;
    int32_t wide;                 // blocks of up to 128 rows on the fp16 matrix cores (head_dim 128)
    int32_t row_tiles;            // otherwise: 16-row tiles per block (1, 2 or 4)
};
struct PrefillPlan {
    int32_t tokens_per_block, pages_per_split, n_splits, row_tiles;
    bool wide;
};
// Row blocks of 16, 32 or 64 rows (row_tiles 1, 2, 4), or of 128 (wide: head_dim 128, for
// chunks with more rows per KV head than 64).
PrefillPlan plan_prefill(int32_t n_tokens, int32_t n_q_heads, int32_t n_kv_heads, int32_t max_seq_len,
                         int32_t window, bool wide, int32_t row_tiles);
// Whether chunks of about n_tokens / n_seqs tokens take the wide blocks.
inline bool prefill_wide(int32_t n_tokens, int32_t n_seqs, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim) {
    const int64_t per_chunk = ((int64_t)n_tokens + n_seqs - 1) / std::max<int32_t>(1, n_seqs);
    return head_dim == 128 && per_chunk * (n_q_heads / n_kv_heads) > 64;
}
// The 16-row tiles a block of the 64-row kernel takes for chunks of about n_tokens / n_seqs
// tokens (blocks then hold that many rows at most: longer chunks get more blocks).
inline int32_t prefill_row_tiles(int32_t n_tokens, int32_t n_seqs, int32_t n_q_heads, int32_t n_kv_heads) {
    const int64_t per_chunk = ((int64_t)n_tokens + n_seqs - 1) / std::max<int32_t>(1, n_seqs);
    const int64_t rows = per_chunk * (n_q_heads / n_kv_heads);
    return rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
}
hipError_t launch_prefill(const PrefillArgs& a, int d, int2* row_blocks, int32_t* n_row_blocks, hipStream_t st);

}  // namespace oaken
