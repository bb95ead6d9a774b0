// Chunked-prefill attention over the quantized cache (the prefill stage also reads the KV
// cache, Sec. 2.1; the sliding window of Sec. 6.1 applies per query).
//
// A workgroup takes a block of 16, 32 or 64 query rows (sized to the mean chunk; longer
// chunks take several blocks): consecutive query tokens of one sequence's chunk times the
// query heads of one KV head.  It reads every page of the
// keys those rows can see once, whatever the number of rows: each page record is staged
// in LDS, dequantized into an fp32 tile (middle values from the dense nibbles, looked up
// in a per-page table of each slot's 16 possible readings, then the COO entries overwrite
// their elements with their true values: the engine's zero-insert and merge of Sec. 5.2),
// and the tile is contracted with all rows on the matrix cores in fp32
// (v_mfma_f32_16x16x4_f32), with an online softmax across the pages (scores in base-2
// units; pages that every row sees skip the masks).  Long prefixes are split into page
// ranges whose partials the decode attention's log-sum-exp combine merges.
//
// The four waves split the channels: each forms every row's partial scores over a quarter
// of the key channels (the partials meet in LDS) and, after the softmax (which every wave
// computes), the outputs of a quarter of the value channels, so the matrix-core work is
// shared evenly whatever the number of rows.  Record bytes are requested two pages ahead
// of the page being processed.  MFMA operand layout (16x16x4, fp32): lane l holds
// A[l & 15][k] and B[k][l & 15] with k = l >> 4 of each 4-wide step; the result holds rows
// 4 (l >> 4) .. + 3 of column l & 15.  Contraction indices are assigned so that a lane's
// operands are contiguous in LDS: step s of lane group g takes channel (d / 16) g + s of
// the wave's quarter of the scores and token 4 g + s of the value product.  Both products
// are formed transposed (keys and values as the A operand, queries and probabilities as
// B), so a query row lives on the four lanes q + 16 g of column q.
//
// With more rows per KV head than one block of 64 holds at head_dim 128 (several query
// heads times a long chunk), prefill_wide_kernel takes up to 128 rows: each wave owns 32
// rows over all the channels, and the tiles are contracted on the fp16 matrix cores with
// every real operand split into a high and a low fp16 part (x = hi + lo to about 2^-22
// relative; the query is fp16 already): S^T = K_hi Q^T + K_lo Q^T and
// O^T += V_hi P_hi + V_hi P_lo + V_lo P_hi, accumulated in fp32.  A page is then read and
// dequantized once for all the rows.
#include "oaken_internal.h"
#include "prefill_internal.h"

#include <hip/hip_fp16.h>

namespace oaken {
namespace {

constexpr int kPfThreads = 256;

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float h2f(uint32_t b) { return __half2float(__ushort_as_half((uint16_t)b)); }

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Maximum and sum over the lane pairs q, q ^ 16 and then q, q ^ 32 (the four lanes q + 16 g
// hold the four quarters of one query row's scores).  v_permlane16_swap with both operands
// v returns the even rows' values in one result and the odd rows' in the other, so their
// combination is the pair's (likewise for the halves and v_permlane32_swap).
__device__ __forceinline__ float max4(float v) {
    const int x = __float_as_int(v);
    const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    const int y = __float_as_int(fmaxf(__int_as_float(a[0]), __int_as_float(a[1])));
    const auto b = __builtin_amdgcn_permlane32_swap(y, y, false, false);
    return fmaxf(__int_as_float(b[0]), __int_as_float(b[1]));
}
__device__ __forceinline__ float sum4(float v) {
    const int x = __float_as_int(v);
    const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    const int y = __float_as_int(__int_as_float(a[0]) + __int_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(y, y, false, false);
    return __int_as_float(b[0]) + __int_as_float(b[1]);
}

// Offsets of a record's fields and its staging area (the COO stream is staged right after
// the counts, metadata, dense nibbles and, with on-demand sparse pages, the page table).
template <int D, bool PG>
struct PfLayout {
    static constexpr Layout LY = PG ? make_layout_paged(kPage, D) : make_layout(kPage, D);
    static constexpr int NC = D / 64;
    static constexpr int NT = kPage * D / kSparsePage;               // page-table entries
    static constexpr int PRE = (int)LY.sparse + (PG ? 4 * NT : 0);   // staged prefix bytes
    static constexpr int CAP = kPage * D;                            // COO capacity
    static constexpr int STAGE = PRE + CAP;
};

constexpr int kWaves = kPfThreads / 64;

// What every prefill kernel stages per page: the two records' bytes, the per-slot
// dequantization constants, the COO bytes used and each COO byte's (slot, chunk) bucket.
template <int D, bool PG>
struct PfStage {
    float tokc[2][kPage][8];                         // per record (K, V) and slot: Min, Delta of
                                                     // inner, middle, outer
    int used[2];                                     // COO bytes of each record
    uint32_t mid[2][kPage][16];                      // per record, slot and nibble: the middle
                                                     // reading in the tiles' word format
    __align__(16) uint8_t rec[2][PfLayout<D, PG>::STAGE];
    uint8_t owner[2][PfLayout<D, PG>::CAP];          // per COO byte: its (slot, chunk) bucket
};

// The dequantized page as fp32 tiles: keys token-major, values channel-major.
template <int D>
struct TilesF32 {
    __align__(16) float kt[kPage][D + 4];
    __align__(16) float vt[D][kPage + 4];
    __device__ void put_k(int t, int j, float x) { kt[t][j] = x; }
    __device__ void put_v(int j, int t, float x) { vt[j][t] = x; }
    // a tile element as one 32-bit word: the fp32 bits
    static __device__ uint32_t word(float x) { return __float_as_uint(x); }
    __device__ void put_k8w(int t, int j0, const uint32_t (&w)[8]) {
        *reinterpret_cast<uint4*>(&kt[t][j0]) = make_uint4(w[0], w[1], w[2], w[3]);
        *reinterpret_cast<uint4*>(&kt[t][j0 + 4]) = make_uint4(w[4], w[5], w[6], w[7]);
    }
    __device__ void put_v8w(int j, int t0, const uint32_t (&w)[8]) {
        *reinterpret_cast<uint4*>(&vt[j][t0]) = make_uint4(w[0], w[1], w[2], w[3]);
        *reinterpret_cast<uint4*>(&vt[j][t0 + 4]) = make_uint4(w[4], w[5], w[6], w[7]);
    }
};

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

// x = hi + lo with both parts fp16: hi the nearest fp16, lo the nearest fp16 to the exact
// rest (about 2^-22 |x| off in all).
struct Split16 {
    _Float16 hi, lo;
};
__device__ __forceinline__ Split16 split16(float x) {
    const _Float16 hi = (_Float16)x;
    return Split16{hi, (_Float16)(x - (float)hi)};
}

// The dequantized page as fp16 high and low parts: key rows of 272 bytes (16-byte aligned
// operand reads, rows spread over the banks), value channel rows of 40 bytes.
template <int D>
struct TilesF16 {
    static constexpr int KS = D + 8, VS = kPage + 4;
    __align__(16) _Float16 kh[kPage][KS];
    __align__(16) _Float16 kl[kPage][KS];
    __align__(16) _Float16 vh[D][VS];
    __align__(16) _Float16 vl[D][VS];
    __device__ void put_k(int t, int j, float x) {
        const Split16 z = split16(x);
        kh[t][j] = z.hi;
        kl[t][j] = z.lo;
    }
    __device__ void put_v(int j, int t, float x) {
        const Split16 z = split16(x);
        vh[j][t] = z.hi;
        vl[j][t] = z.lo;
    }
    // a tile element as one 32-bit word: the high part in the low half, the low part above
    static __device__ uint32_t word(float x) {
        const Split16 z = split16(x);
        return (uint32_t)__builtin_bit_cast(uint16_t, z.hi) | ((uint32_t)__builtin_bit_cast(uint16_t, z.lo) << 16);
    }
    // eight words: their low halves to the high tile, their high halves to the low one
    static __device__ void halves8(const uint32_t (&w)[8], uint4& hi, uint4& lo) {
        hi = make_uint4(__builtin_amdgcn_perm(w[1], w[0], 0x05040100u), __builtin_amdgcn_perm(w[3], w[2], 0x05040100u),
                        __builtin_amdgcn_perm(w[5], w[4], 0x05040100u), __builtin_amdgcn_perm(w[7], w[6], 0x05040100u));
        lo = make_uint4(__builtin_amdgcn_perm(w[1], w[0], 0x07060302u), __builtin_amdgcn_perm(w[3], w[2], 0x07060302u),
                        __builtin_amdgcn_perm(w[5], w[4], 0x07060302u), __builtin_amdgcn_perm(w[7], w[6], 0x07060302u));
    }
    __device__ void put_k8w(int t, int j0, const uint32_t (&w)[8]) {
        uint4 hi, lo;
        halves8(w, hi, lo);
        *reinterpret_cast<uint4*>(&kh[t][j0]) = hi;
        *reinterpret_cast<uint4*>(&kl[t][j0]) = lo;
    }
    __device__ void put_v8w(int j, int t0, const uint32_t (&w)[8]) {
        uint4 hi, lo;
        halves8(w, hi, lo);
        *reinterpret_cast<uint2*>(&vh[j][t0]) = make_uint2(hi.x, hi.y);
        *reinterpret_cast<uint2*>(&vh[j][t0 + 4]) = make_uint2(hi.z, hi.w);
        *reinterpret_cast<uint2*>(&vl[j][t0]) = make_uint2(lo.x, lo.y);
        *reinterpret_cast<uint2*>(&vl[j][t0 + 4]) = make_uint2(lo.z, lo.w);
    }
};

template <int D, bool PG, int RT>
struct PfSmem {
    PfStage<D, PG> st;
    TilesF32<D> tl;
    f4 sp[kWaves][RT][64];                           // per wave: partial scores over its channels
};
template <int D, bool PG>
struct PfWideSmem {
    PfStage<D, PG> st;
    TilesF16<D> tl[2];   // the page being contracted and the next page being dequantized
};

// The record bytes a thread prefetches for the next page: chunk c of record w holds bytes
// [16 c, 16 c + 16) of the record's prefix, or of its COO stream past the prefix.  Fixed
// records also take the first WIN stream bytes in the same pass (the stream follows the
// dense nibbles); with on-demand sparse pages the stream is read once the page table is in.
template <int D, bool PG>
struct PfPrefetch {
    static constexpr int WIN = PG ? 0 : (D == 128 ? 256 : 128);
    static constexpr int CH = PfLayout<D, PG>::PRE / 16 + WIN / 16;   // chunks per record
};

// The dequantization of a page in three phases, every thread of the workgroup taking
// part in each; the page's records are already staged in S.rec (phase 1) and block b is
// valid.  A barrier must separate the phases (pf_dequant_page places them; the 128-row
// kernel interleaves its own work with them).
// (2) buckets, per-slot constants and the middle-reading table
template <int D, bool PG, class Tiles>
__device__ __forceinline__ void pf_phase_buckets(PfStage<D, PG>& S, const float (&tk)[4], const float (&tv)[4],
                                                 int tid) {
    using PL = PfLayout<D, PG>;
    constexpr Layout LY = PL::LY;
    constexpr int NC = PL::NC;
    const int lane = tid & 63, wave = tid >> 6;
    // (2) wave 0: each record's (slot, chunk) buckets, their stream offsets (a DPP prefix
    //     sum: K buckets on lanes 0.., V buckets on lanes 32..) and the bucket owning each
    //     stream byte; wave 1: per-slot dequantization constants
    if (wave == 0) {
        const int w = lane >> 5, bk = lane & 31;
        const int cnt = bk < kPage * NC ? (int)S.rec[w][LY.counts + bk] : 0;
        int x = cnt;
        x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
        x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
        x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
        x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
        x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);   // row_bcast:15 into rows 1, 3
        const int st = x - cnt;
        if (bk == 31) S.used[w] = min(x, PL::CAP);
        for (int k = 0; k < cnt && st + k < PL::CAP; ++k) S.owner[w][st + k] = (uint8_t)bk;
    } else if (wave == 1 && lane < 2 * kPage) {
        const int w = lane / kPage, t = lane % kPage;
        const uint16_t* mt = reinterpret_cast<const uint16_t*>(S.rec[w] + LY.meta + 12 * t);
#pragma unroll
        for (int k = 0; k < 6; ++k) S.tokc[w][t][k] = h2f(mt[k]);
    }
    // the middle reading of each (record, slot, nibble): offset-binary code u, side u >= 8
    // (Eq. 3 inverted, then the Eq. 4 shift undone), in the tiles' word format
#pragma unroll
    for (int i = 0; i < 2 * kPage * 16 / kPfThreads; ++i) {
        const int e = tid + i * kPfThreads, w = e / (kPage * 16), t = (e / 16) % kPage, u = e % 16;
        const uint16_t* mt = reinterpret_cast<const uint16_t*>(S.rec[w] + LY.meta + 12 * t);
        const float mn = h2f(mt[2]), dl = h2f(mt[3]);
        // (thresholds selected as values: an array picked by pointer would live in scratch)
        const float th_lo = w ? tv[1] : tk[1], th_hi = w ? tv[2] : tk[2];
        const bool hi = u >= 8;
        const float mag = mn + (float)(hi ? u - 8 : 7 - u) * dl;
        S.mid[w][t][u] = Tiles::word(hi ? th_hi + mag : th_lo - mag);
    }
}

// (3) the stream bytes past the prefetched window, and the middle readings into the tiles
template <int D, bool PG, class Tiles>
__device__ __forceinline__ void pf_phase_middle(PfStage<D, PG>& S, Tiles& T, const PrefillArgs& a, int b, int h,
                                                int tid) {
    using PL = PfLayout<D, PG>;
    using PF = PfPrefetch<D, PG>;
    constexpr Layout LY = PL::LY;
    auto record = [&](int w) { return a.pool + (((int64_t)b * a.H + h) * 2 + w) * a.stride; };
    // (3) stream bytes past the prefetched window (and, with on-demand sparse pages, the
    //     whole stream, through the page table)
    if (PG || S.used[0] > PF::WIN || S.used[1] > PF::WIN) {
        const int c0 = PF::WIN / 16;
        const int nk = max(0, (S.used[0] + 15) / 16 - c0), nv = max(0, (S.used[1] + 15) / 16 - c0);
        for (int c = tid; c < nk + nv; c += kPfThreads) {
            const int w = c >= nk, cc = c0 + (c - w * nk);
            const uint8_t* src;
            if constexpr (PG) {
                const int32_t e = reinterpret_cast<const int32_t*>(S.rec[w] + LY.sparse)[(16 * cc) / kSparsePage] - 1;
                src = a.spool + (int64_t)((e >= 0 && e < a.spages) ? e : 0) * kSparsePage + (16 * cc) % kSparsePage;
            } else {
                src = record(w) + LY.sparse + 16 * cc;
            }
            *reinterpret_cast<uint4*>(&S.rec[w][PL::PRE + 16 * cc]) = *reinterpret_cast<const uint4*>(src);
        }
    }
    // middle reading of every nibble into the tiles
    {
        // keys: thread = (slot, 8 channels); dense byte t * d/2 + j/2, low nibble = even j
        constexpr int GPT = D / 8;
        if (tid < kPage * GPT) {
            const int t = tid / GPT, cg = tid % GPT;
            const uint32_t dw = *reinterpret_cast<const uint32_t*>(&S.rec[0][LY.dense + t * (D / 2) + 4 * cg]);
            uint32_t x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = S.mid[0][t][(dw >> (4 * e)) & 15u];
            T.put_k8w(t, 8 * cg, x);
        }
        // values: thread = (channel j, 8 slots); dense byte j * 8 + t/2, low nibble = even t
        if (tid < 2 * D) {
            const int j = tid >> 1, t0 = 8 * (tid & 1);
            const uint32_t dw = *reinterpret_cast<const uint32_t*>(&S.rec[1][LY.dense + j * (kPage / 2) + (t0 >> 1)]);
            uint32_t x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = S.mid[1][t0 + e][(dw >> (4 * e)) & 15u];
            T.put_v8w(j, t0, x);
        }
    }
}

// (4) the COO entries' true values into the tiles
template <int D, bool PG, class Tiles>
__device__ __forceinline__ void pf_phase_entries(PfStage<D, PG>& S, Tiles& T, const float (&tk)[4],
                                                 const float (&tv)[4], int tid) {
    using PL = PfLayout<D, PG>;
    constexpr Layout LY = PL::LY;
    constexpr int NC = PL::NC;
    // (4) COO entries replace their elements' middle readings by their true values
    //     (thread = entry of either record's stream)
    {
        const int uk = S.used[0], utot = uk + S.used[1];
        for (int e = tid; e < utot; e += kPfThreads) {
            const int w = e >= uk, ee = e - w * uk;
            const uint8_t* r = S.rec[w];
            const int bk = S.owner[w][ee], t = bk / NC, c = bk % NC;
            const uint32_t en = r[PL::PRE + ee];
            const int j = 64 * c + (int)(en & 63u);
            const uint32_t byte = w ? r[LY.dense + j * (kPage / 2) + (t >> 1)] : r[LY.dense + t * (D / 2) + (j >> 1)];
            const uint32_t n = (byte >> (4 * (w ? (t & 1) : (j & 1)))) & 15u;
            const bool side = (en >> 7) != 0, outer = ((en >> 6) & 1u) != 0;
            const float th_lo = w ? tv[0] : tk[0], th_hi = w ? tv[3] : tk[3];
            const float cf = (float)(side ? n : 15u - n);
            const float mag = outer ? S.tokc[w][t][4] + cf * S.tokc[w][t][5] : S.tokc[w][t][0] + cf * S.tokc[w][t][1];
            const float x = outer ? (side ? th_hi + mag : th_lo - mag) : (side ? mag : -mag);
            if (w) T.put_v(j, t, x);
            else T.put_k(t, j, x);
        }
    }
}

// Phases (2)-(4) with their barriers: leaves the dequantized page in the tiles.
template <int D, bool PG, class Tiles>
__device__ __forceinline__ void pf_dequant_page(PfStage<D, PG>& S, Tiles& T, const PrefillArgs& a, int b, int h,
                                                const float (&tk)[4], const float (&tv)[4], int tid) {
    pf_phase_buckets<D, PG, Tiles>(S, tk, tv, tid);
    __syncthreads();
    pf_phase_middle<D, PG, Tiles>(S, T, a, b, h, tid);
    __syncthreads();
    pf_phase_entries<D, PG, Tiles>(S, T, tk, tv, tid);
    __syncthreads();
}

// The row block's pages [pg_first, pg_end) and its rows' positions (shared by both kernels).
struct PfBlock {
    int s, i0, tok0, C, start, G, i_end, n_rows, pg_first, pg_end;
};
__device__ __forceinline__ PfBlock pf_block(const PrefillArgs& a, int split) {
    PfBlock B;
    const int2 blk = a.row_blocks[blockIdx.x];
    B.s = blk.x;
    B.i0 = blk.y;
    B.tok0 = a.cu_tokens[B.s];
    B.C = a.cu_tokens[B.s + 1] - B.tok0;
    B.start = a.start_pos[B.s];
    B.G = a.Hq / a.H;
    B.i_end = min(B.C, B.i0 + a.tokens_per_block);
    B.n_rows = max(0, (B.i_end - B.i0) * B.G);
    const int p_last = B.start + B.i_end - 1;
    const int lo_first = a.window > 0 ? max(0, B.start + B.i0 + 1 - a.window) : 0;
    B.pg_first = lo_first / kPage + split * a.pages_per_split;
    B.pg_end = min(p_last / kPage + 1, lo_first / kPage + (split + 1) * a.pages_per_split);
    return B;
}

// RT 16-row tiles per block (1, 2 or 4): registers and LDS sized for them, so that short
// chunks get more workgroups per CU.
template <int D, bool PG, int RT>
__global__ __launch_bounds__(kPfThreads) __attribute__((amdgpu_waves_per_eu(RT == 1 ? 4 : 3))) void prefill_kernel(
    PrefillArgs a) {
    using PL = PfLayout<D, PG>;
    using PF = PfPrefetch<D, PG>;
    constexpr int CPW = D / kWaves;    // channels of each wave (scores and outputs)
    constexpr int KSW = CPW / 4;       // 4-wide contraction steps of a wave's scores
    constexpr int NCT = CPW / 16;      // 16-wide output tiles of a wave
    static_assert(PL::PRE % 16 == 0 && 2 * PF::CH <= kPfThreads, "one prefetch chunk per thread");

    __shared__ PfSmem<D, PG, RT> S;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4;
    if ((int)blockIdx.x >= *a.n_row_blocks) return;   // (uniform)
    const int h = blockIdx.y, split = blockIdx.z;
    const PfBlock Bk = pf_block(a, split);
    const int G = Bk.G, n_rows = Bk.n_rows, tok0 = Bk.tok0, i0 = Bk.i0, start = Bk.start;
    const int R = (n_rows + 15) / 16;                 // 16-row tiles
    const int pg_first = Bk.pg_first, pg_end = Bk.pg_end;
    const float* th = a.thr + h * 8;
    const float tk[4] = {th[0], th[1], th[2], th[3]}, tv[4] = {th[4], th[5], th[6], th[7]};

    // ---- rows ------------------------------------------------------------------------
    // Scores are kept in base-2 units (scaled by log2 e, so that the softmax exponentials
    // are single exp2 instructions); the partials' maxima go out in natural units.
    const float sl2 = a.scale * 1.44269504088896341f;
    // pages whose every key every row of the block sees need no mask
    const int vis_hi = start + i0;
    const int vis_lo = a.window > 0 ? max(0, start + Bk.i_end - a.window) : 0;
    // Transposed products: scores S^T = K Q^T and outputs O^T = V^T P^T, so that the lanes
    // holding a query row's scores (column lane & 15 of the result) also hold its
    // probabilities as the B operand of the value product and its outputs, and the softmax
    // state of that row.  B operand (queries, scaled): row tile rt, query row lane & 15,
    // this wave's channels CPW w + KSW g + k.
    float bq[RT][KSW];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int ra = 16 * rt + (lane & 15);
        const bool ok = ra < n_rows;
        const int i = i0 + (ok ? ra / G : 0), hd = ok ? ra % G : 0;
        const uint16_t* qp = a.q + ((int64_t)(tok0 + i) * a.Hq + h * G + hd) * D + CPW * wave + KSW * g;
#pragma unroll
        for (int k = 0; k < KSW; ++k) bq[rt][k] = ok ? sl2 * h2f(qp[k]) : 0.0f;
    }
    // this lane's query row in each tile, its position and window start
    int rpos[RT], rlo[RT];
    bool rok[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int rc = 16 * rt + (lane & 15);
        rok[rt] = rc < n_rows;
        rpos[rt] = start + i0 + (rok[rt] ? rc / G : 0);
        rlo[rt] = a.window > 0 ? max(0, rpos[rt] + 1 - a.window) : 0;
    }
    float m[RT], l[RT];
    f4 o[RT][NCT];   // O^T: channels CPW w + 16 n + 4 g + r of the lane's query row
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        m[rt] = -INFINITY;
        l[rt] = 0.0f;
#pragma unroll
        for (int n = 0; n < NCT; ++n) o[rt][n] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }

    const int32_t* btab = a.block_table + (int64_t)Bk.s * a.max_blocks;
    auto record = [&](int b, int w) { return a.pool + (((int64_t)b * a.H + h) * 2 + w) * a.stride; };
    auto valid_block = [&](int b) { return b >= 0 && b < a.num_blocks; };
    const int pw_ = tid / PF::CH, pc_ = tid % PF::CH;   // this thread's prefetch chunk
    auto prefetch = [&](int pg) -> uint4 {
        if (pg >= pg_end || tid >= 2 * PF::CH) return make_uint4(0, 0, 0, 0);
        const int b = btab[pg];
        if (!valid_block(b)) return make_uint4(0, 0, 0, 0);
        return *reinterpret_cast<const uint4*>(record(b, pw_) + 16 * pc_);
    };

    // One set of tiles and one staging area, with the next page's bucket phase overlapped:
    // once a page's partial scores are out, its records are no longer read, so the next
    // page is staged and its buckets, constants and table are formed while this page's
    // softmax and value product run.
    uint4 cur = prefetch(pg_first), nxt = prefetch(pg_first + 1);
    bool ok_cur = false;   // (uniform) the page in the tiles is valid
    if (pg_first < pg_end) {
        const int b = btab[pg_first];
        if (tid < 2 * PF::CH) *reinterpret_cast<uint4*>(&S.st.rec[pw_][16 * pc_]) = cur;
        cur = nxt;
        nxt = prefetch(pg_first + 2);
        __syncthreads();
        ok_cur = valid_block(b);   // (a precondition violation reads nothing)
        if (ok_cur) pf_dequant_page<D, PG>(S.st, S.tl, a, b, h, tk, tv, tid);
    }
    for (int pg = pg_first; pg < pg_end; ++pg) {
        const bool has_next = pg + 1 < pg_end;
        const int bn = has_next ? btab[pg + 1] : -1;
        const bool ok_next = has_next && valid_block(bn);
        const bool full = pg * kPage + kPage - 1 <= vis_hi && pg * kPage >= vis_lo;

        // (5) partial scores of every row tile over this wave's channels: lane (g, query
        //     row q) gets S^T[4 g + r][q] over channels CPW w .. + CPW
        if (ok_cur) {
            const float* krow = &S.tl.kt[lane & 15][CPW * wave + KSW * g];
            float ka[KSW];
#pragma unroll
            for (int k = 0; k < KSW; k += 4) {
                const float4 v = *reinterpret_cast<const float4*>(krow + k);
                ka[k] = v.x; ka[k + 1] = v.y; ka[k + 2] = v.z; ka[k + 3] = v.w;
            }
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                if (rt >= R) break;
                f4 sc = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int k = 0; k < KSW; ++k) sc = mfma4(ka[k], bq[rt][k], sc);
                S.sp[wave][rt][lane] = sc;
            }
        }
        // (1) stage the next page's prefetched bytes, request the bytes three pages ahead
        if (has_next && tid < 2 * PF::CH) *reinterpret_cast<uint4*>(&S.st.rec[pw_][16 * pc_]) = cur;
        cur = nxt;
        nxt = prefetch(pg + 3);
        __syncthreads();
        // (2) the next page's buckets, constants and middle-reading table
        if (ok_next) pf_phase_buckets<D, PG, TilesF32<D>>(S.st, tk, tv, tid);

        if (ok_cur) {
            // (6) whole scores (the waves' partials summed), online softmax of the lane's query
            //     row over the page's 16 keys (four here, the other twelve on lanes +-16, +-32),
            //     then the value product over this wave's output channels
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                if (rt >= R) break;
                f4 sc = S.sp[0][rt][lane];
#pragma unroll
                for (int w = 1; w < kWaves; ++w) sc += S.sp[w][rt][lane];
                float v[4];
                if (full) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[r] = sc[r];
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int kp = pg * kPage + 4 * g + r;   // key position
                        const bool vis = rok[rt] && kp <= rpos[rt] && kp >= rlo[rt];
                        v[r] = vis ? sc[r] : -INFINITY;
                    }
                }
                const float mx = max4(fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
                const float mn = fmaxf(m[rt], mx);
                // (a row with no visible key yet keeps l = 0 and o = 0 whatever alpha is)
                const float ms = (mn == -INFINITY) ? 0.0f : mn;
                const float alpha = __builtin_amdgcn_exp2f(m[rt] - ms);
                float p[4], ps = 0.0f;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    p[r] = __builtin_amdgcn_exp2f(v[r] - ms);
                    ps += p[r];
                }
                ps = sum4(ps);
                l[rt] = l[rt] * alpha + ps;
                m[rt] = mn;
                // (the accumulators are rescaled only when some row's maximum moved)
                if (__builtin_amdgcn_ballot_w64(alpha != 1.0f)) {
#pragma unroll
                    for (int n = 0; n < NCT; ++n) o[rt][n] *= alpha;
                }
                // O^T += V^T P^T: A = the value tile's channels (row) x tokens 4 g + s, B = this
                // lane's probabilities
#pragma unroll
                for (int n = 0; n < NCT; ++n) {
                    const float4 va =
                        *reinterpret_cast<const float4*>(&S.tl.vt[CPW * wave + 16 * n + (lane & 15)][4 * g]);
                    o[rt][n] = mfma4(va.x, p[0], o[rt][n]);
                    o[rt][n] = mfma4(va.y, p[1], o[rt][n]);
                    o[rt][n] = mfma4(va.z, p[2], o[rt][n]);
                    o[rt][n] = mfma4(va.w, p[3], o[rt][n]);
                }
            }
        }
        __syncthreads();
        // (3), (4) the next page's middle readings and COO entries into the tiles
        if (ok_next) pf_phase_middle<D, PG, TilesF32<D>>(S.st, S.tl, a, bn, h, tid);
        __syncthreads();
        if (ok_next) pf_phase_entries<D, PG, TilesF32<D>>(S.st, S.tl, tk, tv, tid);
        __syncthreads();
        ok_cur = ok_next;
    }

    // ---- outputs (this wave's channels), or this range's partials ------------------------
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        if (rt >= R || !rok[rt]) continue;
        const int rc = 16 * rt + (lane & 15);
        const int64_t row = (int64_t)(tok0 + i0 + rc / G) * a.Hq + h * G + rc % G;
        if (a.n_splits == 1) {
            const float inv = l[rt] > 0.0f ? 1.0f / l[rt] : 0.0f;
#pragma unroll
            for (int n = 0; n < NCT; ++n)
                *reinterpret_cast<float4*>(&a.out[row * D + CPW * wave + 16 * n + 4 * g]) =
                    make_float4(o[rt][n][0] * inv, o[rt][n][1] * inv, o[rt][n][2] * inv, o[rt][n][3] * inv);
        } else {
            float* pp = a.partial + (row * a.n_splits + split) * (D + 2);
#pragma unroll
            for (int n = 0; n < NCT; ++n)
                for (int r = 0; r < 4; ++r) pp[CPW * wave + 16 * n + 4 * g + r] = o[rt][n][r];
            if (wave == 0 && g == 0) {
                pp[D] = m[rt] * 0.693147180559945309f;
                pp[D + 1] = l[rt];
            }
        }
    }
}

// Up to kWideRows rows per block: wave w owns rows 32 w .. 32 w + 31 (two row tiles) over all
// D channels.  Per page and row tile: S^T = K Q^T on v_mfma_f32_16x16x32_f16 (A = 8 fp16 of
// a key row, K_hi then K_lo; B = the row's query, unscaled fp16), the online softmax as in
// prefill_kernel (scale applied to the fp32 scores), then O^T += V^T P^T on
// v_mfma_f32_16x16x16f16 with P split into hi and lo in registers.  The key and value
// operands read from LDS serve all four row tiles of the wave.
constexpr int kWideRows = 128;
constexpr int kWideTiles = kWideRows / kWaves / 16;   // row tiles per wave

template <bool PG>
__global__ __launch_bounds__(kPfThreads) __attribute__((amdgpu_waves_per_eu(3))) void prefill_wide_kernel(PrefillArgs a) {
    constexpr int D = 128;
    using PL = PfLayout<D, PG>;
    using PF = PfPrefetch<D, PG>;
    constexpr int NCT = D / 16;        // output channel tiles
    constexpr int KST = D / 32;        // 32-wide contraction steps of the scores
    static_assert(PL::PRE % 16 == 0 && 2 * PF::CH <= kPfThreads, "one prefetch chunk per thread");

    __shared__ PfWideSmem<D, PG> S;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, q16 = lane & 15;
    if ((int)blockIdx.x >= *a.n_row_blocks) return;   // (uniform)
    const int h = blockIdx.y, split = blockIdx.z;
    const PfBlock Bk = pf_block(a, split);
    const int G = Bk.G, tok0 = Bk.tok0, i0 = Bk.i0, start = Bk.start;
    const int wrow0 = kWideTiles * 16 * wave;                          // the wave's first row
    const int R = max(0, min(kWideTiles, (Bk.n_rows - wrow0 + 15) / 16));   // its row tiles
    const int pg_first = Bk.pg_first, pg_end = Bk.pg_end;
    const float* th = a.thr + h * 8;
    const float tk[4] = {th[0], th[1], th[2], th[3]}, tv[4] = {th[4], th[5], th[6], th[7]};

    // B operand of the scores: row tile rt, query row q16, channels 32 k + 8 g .. + 7
    h8 bq[kWideTiles][KST];
    int rpos[kWideTiles], rlo[kWideTiles];
    bool rok[kWideTiles];
#pragma unroll
    for (int rt = 0; rt < kWideTiles; ++rt) {
        const int rc = wrow0 + 16 * rt + q16;
        rok[rt] = rc < Bk.n_rows;
        const int i = i0 + (rok[rt] ? rc / G : 0), hd = rok[rt] ? rc % G : 0;
        const uint16_t* qp = a.q + ((int64_t)(tok0 + i) * a.Hq + h * G + hd) * D + 8 * g;
#pragma unroll
        for (int k = 0; k < KST; ++k) {
            const uint4 w = rok[rt] ? *reinterpret_cast<const uint4*>(qp + 32 * k) : make_uint4(0, 0, 0, 0);
            bq[rt][k] = __builtin_bit_cast(h8, w);
        }
        rpos[rt] = start + i;
        rlo[rt] = a.window > 0 ? max(0, rpos[rt] + 1 - a.window) : 0;
    }
    // scores in base-2 units (see prefill_kernel); pages every row sees need no mask
    const float sl2 = a.scale * 1.44269504088896341f;
    const int vis_hi = start + i0;
    const int vis_lo = a.window > 0 ? max(0, start + Bk.i_end - a.window) : 0;
    float m[kWideTiles], l[kWideTiles];
    f4 o[kWideTiles][NCT];   // O^T: channels 16 n + 4 g + r of the lane's query row
#pragma unroll
    for (int rt = 0; rt < kWideTiles; ++rt) {
        m[rt] = -INFINITY;
        l[rt] = 0.0f;
#pragma unroll
        for (int n = 0; n < NCT; ++n) o[rt][n] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }

    const int32_t* btab = a.block_table + (int64_t)Bk.s * a.max_blocks;
    auto record = [&](int b, int w) { return a.pool + (((int64_t)b * a.H + h) * 2 + w) * a.stride; };
    auto valid_block = [&](int b) { return b >= 0 && b < a.num_blocks; };
    const int pw_ = tid / PF::CH, pc_ = tid % PF::CH;   // this thread's prefetch chunk
    auto prefetch = [&](int pg) -> uint4 {
        if (pg >= pg_end || tid >= 2 * PF::CH) return make_uint4(0, 0, 0, 0);
        const int b = btab[pg];
        if (!valid_block(b)) return make_uint4(0, 0, 0, 0);
        return *reinterpret_cast<const uint4*>(record(b, pw_) + 16 * pc_);
    };

    // (two pages in flight: with few workgroups per CU one page ahead does not cover the
    // memory latency)
    // Software pipeline over the pages: while the waves contract page pg from one set of
    // tiles, they stage and dequantize page pg + 1 into the other, each wave taking up its
    // share of the next page's phases between its own matrix-core and softmax steps, so
    // that the barriers between the phases find work to overlap.
    uint4 cur = prefetch(pg_first), nxt = prefetch(pg_first + 1);
    bool ok_cur = false;   // (uniform) the page in the current tiles is valid
    if (pg_first < pg_end) {
        const int b = btab[pg_first];
        if (tid < 2 * PF::CH) *reinterpret_cast<uint4*>(&S.st.rec[pw_][16 * pc_]) = cur;
        cur = nxt;
        nxt = prefetch(pg_first + 2);
        __syncthreads();
        ok_cur = valid_block(b);   // (a precondition violation reads nothing)
        if (ok_cur) pf_dequant_page<D, PG>(S.st, S.tl[0], a, b, h, tk, tv, tid);
    }
    for (int pg = pg_first; pg < pg_end; ++pg) {
        const int par = (pg - pg_first) & 1;
        TilesF16<D>& Tc = S.tl[par];       // page pg
        TilesF16<D>& Tn = S.tl[par ^ 1];   // page pg + 1
        const bool has_next = pg + 1 < pg_end;
        const int bn = has_next ? btab[pg + 1] : -1;
        const bool ok_next = has_next && valid_block(bn);
        // (1) stage the next page (the previous page's phases are past their last barrier)
        if (has_next && tid < 2 * PF::CH) *reinterpret_cast<uint4*>(&S.st.rec[pw_][16 * pc_]) = cur;
        cur = nxt;
        nxt = prefetch(pg + 3);
        const bool work = ok_cur && R > 0;   // (uniform per wave)
        const bool full = pg * kPage + kPage - 1 <= vis_hi && pg * kPage >= vis_lo;

        // scores of the wave's row tiles: lane (g, q16) gets S^T[4 g + r][q16]
        f4 sc[kWideTiles];
#pragma unroll
        for (int rt = 0; rt < kWideTiles; ++rt) sc[rt] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        if (work) {
#pragma unroll
            for (int k = 0; k < KST; ++k) {
                const h8 ah = *reinterpret_cast<const h8*>(&Tc.kh[q16][32 * k + 8 * g]);
                const h8 al = *reinterpret_cast<const h8*>(&Tc.kl[q16][32 * k + 8 * g]);
#pragma unroll
                for (int rt = 0; rt < kWideTiles; ++rt) {
                    if (rt < R) {
                        sc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bq[rt][k], sc[rt], 0, 0, 0);
                        sc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, bq[rt][k], sc[rt], 0, 0, 0);
                    }
                }
            }
        }
        __syncthreads();
        // (2) the next page's buckets, constants and middle-reading table
        if (ok_next) pf_phase_buckets<D, PG, TilesF16<D>>(S.st, tk, tv, tid);

        // online softmax per row tile, probabilities split for the value product
        h4 ph[kWideTiles], pl[kWideTiles];
        if (work) {
#pragma unroll
            for (int rt = 0; rt < kWideTiles; ++rt) {
                if (rt >= R) break;
                float v[4];
                if (full) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[r] = sl2 * sc[rt][r];
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int kp = pg * kPage + 4 * g + r;   // key position
                        const bool vis = rok[rt] && kp <= rpos[rt] && kp >= rlo[rt];
                        v[r] = vis ? sl2 * sc[rt][r] : -INFINITY;
                    }
                }
                const float mx = max4(fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
                const float mn = fmaxf(m[rt], mx);
                // (a row with no visible key yet keeps l = 0 and o = 0 whatever alpha is)
                const float ms = (mn == -INFINITY) ? 0.0f : mn;
                const float alpha = __builtin_amdgcn_exp2f(m[rt] - ms);
                float ps = 0.0f;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float p = __builtin_amdgcn_exp2f(v[r] - ms);
                    ps += p;
                    const Split16 z = split16(p);
                    ph[rt][r] = z.hi;
                    pl[rt][r] = z.lo;
                }
                ps = sum4(ps);
                l[rt] = l[rt] * alpha + ps;
                m[rt] = mn;
                // (the accumulators are rescaled only when some row's maximum moved)
                if (__builtin_amdgcn_ballot_w64(alpha != 1.0f)) {
#pragma unroll
                    for (int n = 0; n < NCT; ++n) o[rt][n] *= alpha;
                }
            }
        }
        __syncthreads();
        // (3) the next page's middle readings
        if (ok_next) pf_phase_middle<D, PG, TilesF16<D>>(S.st, Tn, a, bn, h, tid);

        // O^T += V^T P^T: A = channels 16 n + q16 x keys 4 g .. + 3 (hi, lo); B = the lane's
        // probabilities (hi, lo); the hi x hi, hi x lo and lo x hi products
        if (work) {
#pragma unroll
            for (int n = 0; n < NCT; ++n) {
                const h4 vh = *reinterpret_cast<const h4*>(&Tc.vh[16 * n + q16][4 * g]);
                const h4 vl = *reinterpret_cast<const h4*>(&Tc.vl[16 * n + q16][4 * g]);
#pragma unroll
                for (int rt = 0; rt < kWideTiles; ++rt) {
                    if (rt < R) {
                        o[rt][n] = __builtin_amdgcn_mfma_f32_16x16x16f16(vh, ph[rt], o[rt][n], 0, 0, 0);
                        o[rt][n] = __builtin_amdgcn_mfma_f32_16x16x16f16(vh, pl[rt], o[rt][n], 0, 0, 0);
                        o[rt][n] = __builtin_amdgcn_mfma_f32_16x16x16f16(vl, ph[rt], o[rt][n], 0, 0, 0);
                    }
                }
            }
        }
        __syncthreads();
        // (4) the next page's COO entries; after the barrier its tiles are complete and this
        //     page's are free for the page after
        if (ok_next) pf_phase_entries<D, PG, TilesF16<D>>(S.st, Tn, tk, tv, tid);
        __syncthreads();
        ok_cur = ok_next;
    }

    // ---- outputs, or this range's partials ------------------------------------------------
#pragma unroll
    for (int rt = 0; rt < kWideTiles; ++rt) {
        if (rt >= R || !rok[rt]) continue;
        const int rc = wrow0 + 16 * rt + q16;
        const int64_t row = (int64_t)(tok0 + i0 + rc / G) * a.Hq + h * G + rc % G;
        if (a.n_splits == 1) {
            const float inv = l[rt] > 0.0f ? 1.0f / l[rt] : 0.0f;
#pragma unroll
            for (int n = 0; n < NCT; ++n)
                *reinterpret_cast<float4*>(&a.out[row * D + 16 * n + 4 * g]) =
                    make_float4(o[rt][n][0] * inv, o[rt][n][1] * inv, o[rt][n][2] * inv, o[rt][n][3] * inv);
        } else {
            float* pp = a.partial + (row * a.n_splits + split) * (D + 2);
#pragma unroll
            for (int n = 0; n < NCT; ++n)
                *reinterpret_cast<float4*>(&pp[16 * n + 4 * g]) =
                    make_float4(o[rt][n][0], o[rt][n][1], o[rt][n][2], o[rt][n][3]);
            if (g == 0) {
                pp[D] = m[rt] * 0.693147180559945309f;
                pp[D + 1] = l[rt];
            }
        }
    }
}

// Row blocks: sequence s's chunk of C_s tokens is cut into ceil(C_s / T) blocks of T
// tokens; block k lists (sequence, first token).  One workgroup, sequences in rounds of
// 1024 with a workgroup prefix sum of the block counts.
__global__ __launch_bounds__(1024) void prefill_blocks_kernel(const int32_t* cu_tokens, int n_seqs, int T,
                                                             int max_row_blocks, int2* row_blocks, int32_t* n_row_blocks) {
    __shared__ int scan[1024];
    int base = 0;
    for (int s0 = 0; s0 < n_seqs; s0 += 1024) {
        const int s = s0 + (int)threadIdx.x;
        const int C = s < n_seqs ? max(0, cu_tokens[s + 1] - cu_tokens[s]) : 0;
        const int nb = (C + T - 1) / T;
        scan[threadIdx.x] = nb;
        __syncthreads();
        for (int d = 1; d < 1024; d <<= 1) {
            const int v = threadIdx.x >= (unsigned)d ? scan[threadIdx.x - d] : 0;
            __syncthreads();
            scan[threadIdx.x] += v;
            __syncthreads();
        }
        const int first = base + scan[threadIdx.x] - nb;
        for (int j = 0; j < nb; ++j)
            if (first + j < max_row_blocks) row_blocks[first + j] = make_int2(s, j * T);
        base += scan[1023];
        __syncthreads();
    }
    if (threadIdx.x == 0) *n_row_blocks = min(base, max_row_blocks);
}

}  // namespace

PrefillPlan plan_prefill(int32_t n_tokens, int32_t n_q_heads, int32_t n_kv_heads, int32_t max_seq_len,
                         int32_t window, bool wide, int32_t row_tiles) {
    PrefillPlan p{};
    const int G = n_q_heads / n_kv_heads;
    p.wide = wide;
    p.row_tiles = wide ? kWideRows / 16 : (row_tiles <= 1 ? 1 : (row_tiles <= 2 ? 2 : 4));
    p.tokens_per_block = std::max(1, (wide ? kWideRows : 16 * p.row_tiles) / G);
    // keys a block can see: its own tokens and everything before them (or a window of W
    // before its first token)
    const int64_t span = window > 0 ? std::min<int64_t>(max_seq_len, (int64_t)window + p.tokens_per_block + kPage)
                                    : max_seq_len;
    const int max_pages = (int)((span + kPage - 1) / kPage) + 1;
    const int64_t units = (int64_t)std::max(1, (n_tokens + p.tokens_per_block - 1) / p.tokens_per_block) * n_kv_heads;
    const int want = (int)std::max<int64_t>(1, (2048 + units - 1) / units);
    p.pages_per_split = std::max(16, (max_pages + want - 1) / want);
    p.n_splits = (max_pages + p.pages_per_split - 1) / p.pages_per_split;
    return p;
}

hipError_t launch_prefill(const PrefillArgs& a, int d, int2* row_blocks, int32_t* n_row_blocks, hipStream_t st) {
    hipLaunchKernelGGL(prefill_blocks_kernel, dim3(1), dim3(1024), 0, st, a.cu_tokens, a.n_seqs, a.tokens_per_block,
                       a.max_row_blocks, row_blocks, n_row_blocks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid(a.max_row_blocks, a.H, a.n_splits);
    const bool pg = a.spool != nullptr;
    if (a.wide) {
        if (d != 128) return hipErrorInvalidValue;
        if (pg)
            hipLaunchKernelGGL(prefill_wide_kernel<true>, grid, dim3(kPfThreads), 0, st, a);
        else
            hipLaunchKernelGGL(prefill_wide_kernel<false>, grid, dim3(kPfThreads), 0, st, a);
        return hipGetLastError();
    }
    if (d != 64 && d != 128) return hipErrorInvalidValue;
    if (a.row_tiles != 1 && a.row_tiles != 2 && a.row_tiles != 4) return hipErrorInvalidValue;
    auto go = [&](auto kernel) { hipLaunchKernelGGL(kernel, grid, dim3(kPfThreads), 0, st, a); };
    if (d == 128) {
        if (pg)
            a.row_tiles == 1 ? go(prefill_kernel<128, true, 1>) : a.row_tiles == 2 ? go(prefill_kernel<128, true, 2>)
                                                                   : go(prefill_kernel<128, true, 4>);
        else
            a.row_tiles == 1 ? go(prefill_kernel<128, false, 1>) : a.row_tiles == 2 ? go(prefill_kernel<128, false, 2>)
                                                                    : go(prefill_kernel<128, false, 4>);
    } else {
        if (pg)
            a.row_tiles == 1 ? go(prefill_kernel<64, true, 1>) : a.row_tiles == 2 ? go(prefill_kernel<64, true, 2>)
                                                                  : go(prefill_kernel<64, true, 4>);
        else
            a.row_tiles == 1 ? go(prefill_kernel<64, false, 1>) : a.row_tiles == 2 ? go(prefill_kernel<64, false, 2>)
                                                                   : go(prefill_kernel<64, false, 4>);
    }
    return hipGetLastError();
}

}  // namespace oaken
