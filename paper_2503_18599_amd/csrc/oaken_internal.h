// Private declarations shared by the translation units of liboaken.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace oaken {

constexpr int kPage = 16;         // tokens per page (block_size)
constexpr int kSparsePage = 256;  // bytes of one on-demand sparse page

// Byte offsets of the fields of one page record (layout in include/oaken.h).
struct Layout {
    int64_t counts, meta, dense, sparse, stride;
};

__host__ __device__ constexpr int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

__host__ __device__ constexpr Layout make_layout(int P, int d) {
    Layout L{};
    L.counts = 0;
    L.meta = round_up((int64_t)P * (d / 64), 16);
    L.dense = round_up(L.meta + (int64_t)P * 12, 16);
    L.sparse = L.dense + (int64_t)P * d / 2;
    L.stride = round_up(L.sparse + (int64_t)P * d, 128);
    return L;
}

// With on-demand sparse pages the record ends in its sparse page table (int32 ids of
// the pages holding its COO stream); `sparse` is then the table's offset.
__host__ __device__ constexpr Layout make_layout_paged(int P, int d) {
    Layout L = make_layout(P, d);
    L.stride = round_up(L.sparse + 4 * ((int64_t)P * d / kSparsePage), 128);
    return L;
}

struct QuantArgs {
    uint8_t* pool;
    const float* thr;             // [H][2][4]
    const uint16_t* k_new;        // fp16 bits [n_tokens][H][d]
    const uint16_t* v_new;
    const int32_t* block_table;   // [n_seqs][max_blocks]
    const int32_t* start_pos;     // [n_seqs]
    const int32_t* cu_tokens;     // [n_seqs + 1]
    int64_t stride;
    int32_t num_blocks, H, max_blocks, n_seqs;
    uint8_t* spool;               // on-demand sparse pages (nullptr: fixed records)
    int32_t* sfree;               // free list: [0] count, [1] overflow flag, [2..] page ids
    int32_t spages;
};

struct CalibArgs {
    const uint16_t* k;            // fp16 bits [R][T][H][d]
    const uint16_t* v;
    float* per_run;               // [R][H][2][3] = lo_o, hi_o, t
    float* thr_out;               // [H][2][4]
    int64_t n, k_o, k_i;          // values per run and order-statistic ranks
    int32_t R, T, H, d;
};

struct AttnArgs {
    const uint8_t* pool;
    const float* thr;             // [H][2][4]
    const uint16_t* q;            // fp16 bits [n_seqs][Hq][d]
    const int32_t* block_table;   // [n_seqs][max_blocks]
    const int32_t* seq_lens;      // [n_seqs]
    float* out;                   // fp32 [n_seqs][Hq][d]
    float* partial;               // [n_seqs][Hq][n_splits][d + 2] when n_splits > 1
    int64_t stride;
    int32_t num_blocks, H, Hq, max_blocks, n_seqs, max_seq_len;
    int32_t pages_per_split, n_splits;
    int32_t window;               // sliding window in tokens (<= 0: the whole sequence)
    float scale;
    const uint8_t* spool;         // on-demand sparse pages (nullptr: fixed records)
    int32_t spages;
    // A KV head's G = Hq / H query heads are split over head_parts workgroups of
    // wave_heads heads each (head_parts * wave_heads = G); set by launch_attention.
    int32_t wave_heads, head_parts;
};

// Attention workgroups form a 1-D grid with the KV head varying fastest, then the part of
// its query heads, then the row, then the page range.  Workgroups are handed to the eight
// XCDs round-robin by linear id, so every XCD receives the same heads of every row and
// range: an equal share of the work even when sequence lengths vary (with the range
// fastest, XCD k would get ranges k and k + 8 of every sequence, and the late ranges exist
// only for long sequences).  Early ranges go out first, so the short or empty last ranges
// fill the tail.  The parts of one KV head are H workgroups apart: with H a multiple of 8
// they run on the same XCD, whose L2 then serves the pages a second part reads.
struct AttnTile {
    int split, h, s, part;
};
__device__ __forceinline__ AttnTile attn_tile(const AttnArgs& a) {
    const uint32_t hv_n = (uint32_t)(a.H * a.head_parts);
    const uint32_t id = blockIdx.x, hs = id / hv_n, hv = id % hv_n;   // the grid fits 31 bits
    return AttnTile{(int)(hs / (uint32_t)a.n_seqs), (int)(hv % (uint32_t)a.H), (int)(hs % (uint32_t)a.n_seqs),
                    (int)(hv / (uint32_t)a.H)};
}
// Workgroups of an attention launch; 0 when the grid would not fit one dimension.
inline uint32_t attn_grid(const AttnArgs& a) {
    const int64_t n = (int64_t)a.n_splits * a.H * a.head_parts * a.n_seqs;
    return (n > 0 && n <= 0x7fffffff) ? (uint32_t)n : 0u;
}

// Log-sum-exp merge of split partials for a.n_seqs * a.Hq rows (attention.hip).
hipError_t launch_combine(const AttnArgs& a, int d, hipStream_t st);

// Split-K plan used by both the workspace query and the launch.
struct SplitPlan {
    int32_t pages_per_split, n_splits;
};
SplitPlan plan_splits(int32_t n_seqs, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                      int32_t max_seq_len);

// Sparse page pool maintenance (sparse_pages.hip).
struct SparseArgs {
    uint8_t* pool;                // dense records
    int64_t stride, table;        // record stride; offset of the record's page table
    int32_t num_blocks, H, cbytes, tbytes;   // counts bytes and table bytes per record
    int32_t* sfree;
    int32_t spages;
};
hipError_t launch_sparse_reset(const SparseArgs& a, hipStream_t st);
hipError_t launch_sparse_release(const SparseArgs& a, const int32_t* block_ids, int n_blocks, hipStream_t st);

hipError_t launch_quantize(const QuantArgs& a, int d, int max_new_per_seq, hipStream_t st);
hipError_t launch_calibrate(const CalibArgs& a, hipStream_t st);
hipError_t launch_attention(const AttnArgs& a, int d, hipStream_t st);

// Streaming-read probe (probe.hip).
struct ProbeArgs {
    const uint8_t* base;
    int64_t record_stride, n_records;
    int32_t chunks;               // 16-byte chunks read from the start of each record (<= 256)
    uint32_t* checksum;           // XOR of every 32-bit word read
    uint32_t total_chunks, magic, shift;   // set by prepare_probe
};
bool prepare_probe(ProbeArgs& a);   // false: more than 2^31 - 1 chunks
hipError_t launch_probe_read(const ProbeArgs& a, hipStream_t st);

// Group-count variants of the quantizer (variants.hip).
struct VariantInfo {
    int32_t n_out, n_in, out_bits, rank_bits, coo_bits, coo_bytes, groups;   // groups == 0: unknown
};
VariantInfo variant_info(int variant);
struct VariantArgs {
    VariantInfo info;
    const uint16_t* x;            // fp16 bits [n][H][d]
    const float* thr8;            // [H][8]
    uint8_t* nib;                 // [n][H][d/2]
    uint8_t* coo;                 // [n][H][d * coo_bytes]
    uint8_t* counts;              // [n][H][d/64]
    uint16_t* meta;               // [n][H][2 * groups] fp16 bits
    int32_t* n_coo;               // [n][H]
    float* out;                   // [n][H][d] (dequantization)
    int32_t n, H;
};
hipError_t launch_variant_quantize(const VariantArgs& a, int d, hipStream_t st);
hipError_t launch_variant_dequantize(const VariantArgs& a, int d, hipStream_t st);

// Matrix-core decode attention (head_dim 128; 1..8 query heads per KV head, taken 1, 2 or 4
// per workgroup).
bool mfma_attention_supported(int d, int G);
int mfma_wave_heads(int G);      // query heads per workgroup for G heads per KV head
int mfma_score_cap(int wave_heads);   // tokens per query head in one workgroup's page range
hipError_t launch_attention_mfma(const AttnArgs& a, hipStream_t st);
hipError_t launch_attention_mfma_paged(const AttnArgs& a, hipStream_t st);   // on-demand sparse pages

}  // namespace oaken
