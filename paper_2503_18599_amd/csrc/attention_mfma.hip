// Decode attention over the Oaken-quantized cache on CDNA4 int8 matrix cores
// (head_dim 128; a workgroup takes 1, 2 or 4 query heads of one KV head, and a KV head
// with more query heads, or a number that is not one of these, is split over several
// workgroups that read the same pages).
//
// Dequantization is split into a dense part that runs on MFMA and a sparse part that
// runs on the vector units, mirroring the paper's dense/sparse split (Sec. 4.5) and
// its dequantization engine (Sec. 5.2):
//
// * Every nibble is first read as a middle value.  A middle value is affine in its
//   code u and its side bit h = u >> 3 (Sec. 4.4):  x = base + u*Delta + h*Gp  with
//   per-token base = lo_i - Min - 7 Delta and Gp = hi_i - lo_i + 2 Min - Delta.  So
//   q.K^ = base*sum(q) + Delta*sum(q_j u_j) + Gp*sum(q_j h_j), and
//   p.V^ = sum(p base) + sum_t (p_t Delta_t) u_tj + sum_t (p_t Gp_t) h_tj.
//   Both reduce to integer contractions of the raw nibble bytes.  Four int8 features
//   per byte (the byte itself, its low nibble, and two bit-3 masks; three VALU
//   operations per eight elements) span u and h of both nibbles, and the real-valued
//   weights (the query, or p*Delta and p*Gp) enter as four balanced base-256 int8
//   limbs.  v_mfma_i32_16x16x64_i8 then computes the sums exactly in int32.
// * Inner and outer values (the COO stream) are corrected afterwards: each entry adds
//   its true value minus the middle reading of its nibble.  One lane walks the entries
//   of one (token, 64-value chunk) bucket; a per-token table gives the correction as
//   an affine function of the nibble for each (group, side) class.
//
// One wave owns (sequence, KV head, page range).  Pass 1 streams the key pages and
// leaves scores in LDS, then the range's softmax, then pass 2 streams the value pages.
// Pages move in groups of four through a software pipeline: while a group is being
// processed, the dense and sparse bytes of the next group and the record heads
// (counts and scales) of the group after it are already in flight, so every sparse
// offset is known before its bytes are requested.
#include "oaken_internal.h"

#include <hip/hip_fp16.h>

namespace oaken {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int D = 128;
constexpr int P = kPage;
constexpr Layout LY = make_layout(P, D);   // counts 0, meta 32, dense 224, sparse 1248
constexpr int HB = 224;                    // counts + meta bytes at the start of a record
constexpr int CB = 32;                     // COO count bytes at the start of a record
constexpr int cmax(int x, int y) { return x > y ? x : y; }
constexpr int GRP = 4;                     // pages per group (two correction pairs)
constexpr int GT = GRP * P;                // tokens per group
// LDS stride of a key page's dense bytes (token rows of 64 bytes).
constexpr int PSTR = 1088;
// Value pages are staged as stored (channel c's dwords of tokens 0-7 and 8-15 at 8c and
// 8c + 4), page q + 2 right after page q, pair q at q * VREG: the two dwords a value MFMA
// lane takes (pages q and q + 2) are then 1024 bytes apart, one two-address read, and
// staging writes the loaded registers unchanged.
constexpr int VREG = 2 * 1024 + 128;
static_assert(2 * VREG <= GRP * PSTR, "value staging fits the dense buffer");
__host__ __device__ constexpr int vpos(int pg) { return (pg & 1) * VREG + (pg >> 1) * 1024; }
constexpr int SPCAP = P * D;               // sparse capacity of one record
constexpr int SSLOT = 448;                 // staged COO bytes per page (larger pages: read from HBM)
constexpr int SPL = GRP * SSLOT;           // group sparse bytes staged in LDS

static_assert(LY.meta == 32 && LY.dense == HB && LY.sparse == 1248, "record layout");

__device__ __forceinline__ float h2f(uint16_t b) { return __half2float(__ushort_as_half(b)); }
__device__ __forceinline__ float fin(float x) { return __builtin_isfinite(x) ? x : 0.0f; }

// Balanced base-256 digits of w (|w| < 2^30): byte r is the int8 digit of limb r.
__device__ __forceinline__ uint32_t enc(int w) {
    return ((uint32_t)w + 0x80808080u) ^ 0x80808080u;
}
__device__ __forceinline__ uint32_t byte_of(uint32_t w, int r) { return (w >> (8 * r)) & 0xffu; }

// The four int8 features of four nibble bytes: raw byte, low nibble, bits 7|3, bit 3.
__device__ __forceinline__ v4i features(uint32_t d) {
    v4i b;
    b[0] = (int)d;
    b[1] = (int)(d & 0x0f0f0f0fu);
    b[2] = (int)(d & 0x88888888u);
    b[3] = (int)(d & 0x08080808u);
    return b;
}

// Feature f of four dwords of nibble bytes (f = 0 the bytes themselves).
__device__ __forceinline__ v4i feature_of(const uint4& d, int f) {
    const uint32_t msk = f == 1 ? 0x0f0f0f0fu : f == 2 ? 0x88888888u : 0x08080808u;
    if (f == 0) return v4i{(int)d.x, (int)d.y, (int)d.z, (int)d.w};
    return v4i{(int)(d.x & msk), (int)(d.y & msk), (int)(d.z & msk), (int)(d.w & msk)};
}

__device__ __forceinline__ v4i mfma(v4i a, v4i b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// Value of four base-256 limbs (each |limb sum| < 2^22: the pairs combine exactly in
// int32 before the two conversions).
__device__ __forceinline__ float limbs(v4i c) {
    const int lo = __mul24(c[1], 256) + c[0], hi = __mul24(c[3], 256) + c[2];
    return fmaf((float)hi, 65536.0f, (float)lo);
}

// Wave reductions: a shift-scan within each row of 16 lanes (DPP row_shr 1, 2, 4, 8
// leaves the row's total in its lane 15), then the four row totals through readlane.
// No LDS round trip; the result is wave-uniform.
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, T ident, Op op) {
    static_assert(sizeof(T) == 4, "32-bit values");
    const int id = __builtin_bit_cast(int, ident);
    v = op(v, __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(id, __builtin_bit_cast(int, v), 0x111, 0xf, 0xf, false)));
    v = op(v, __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(id, __builtin_bit_cast(int, v), 0x112, 0xf, 0xf, false)));
    v = op(v, __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(id, __builtin_bit_cast(int, v), 0x114, 0xf, 0xf, false)));
    v = op(v, __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(id, __builtin_bit_cast(int, v), 0x118, 0xf, 0xf, false)));
    const int x = __builtin_bit_cast(int, v);
    const T r0 = __builtin_bit_cast(T, __builtin_amdgcn_readlane(x, 15));
    const T r1 = __builtin_bit_cast(T, __builtin_amdgcn_readlane(x, 31));
    const T r2 = __builtin_bit_cast(T, __builtin_amdgcn_readlane(x, 47));
    const T r3 = __builtin_bit_cast(T, __builtin_amdgcn_readlane(x, 63));
    return op(op(r0, r1), op(r2, r3));
}
__device__ __forceinline__ float wave_max(float v) {
    return wave_reduce(v, -INFINITY, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ float wave_sum(float v) {
    return wave_reduce(v, 0.0f, [](float a, float b) { return a + b; });
}
// Maximum of non-negative floats (their bit patterns order as unsigned integers); lanes
// shifted in from outside a row read 0.
__device__ __forceinline__ float wave_max_nonneg(float v) {
    uint32_t x = __builtin_bit_cast(uint32_t, v);
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true));
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true));
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true));
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true));
    const uint32_t r = max(max((uint32_t)__builtin_amdgcn_readlane((int)x, 15), (uint32_t)__builtin_amdgcn_readlane((int)x, 31)),
                           max((uint32_t)__builtin_amdgcn_readlane((int)x, 47), (uint32_t)__builtin_amdgcn_readlane((int)x, 63)));
    return __builtin_bit_cast(float, r);
}
__device__ __forceinline__ int wave_max_i(int v) {
    return wave_reduce(v, (int)0x80000000, [](int a, int b) { return max(a, b); });
}

// Inclusive prefix sum within each row of 16 lanes (DPP row shifts).
__device__ __forceinline__ int row_scan16(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
    return x;
}

// Fixed-point shift so that |x| * 2^shift <= 2^22 for every |x| <= mx.
__device__ __forceinline__ int fix_shift(float mx) {
    if (!(mx > 0.0f)) return 0;
    int e;
    frexpf(mx, &e);
    return 22 - e;
}

// Per-token constants of the dequantization (thresholds th = lo_o, lo_i, hi_i, hi_o).
struct Tok {
    float base, dm, gp;   // middle reading: base + u*dm + h*gp
    float b_il, b_ol, b_ih, b_oh, kd_i, kd_o;
};

// The token's 12 metadata bytes (three fp16 pairs Min, Delta: inner, middle, outer).
struct Meta {
    uint32_t w0, w1, w2;
};

__device__ __forceinline__ Tok token_consts(const Meta& mt, const float* th) {
    const uint32_t w0 = mt.w0, w1 = mt.w1, w2 = mt.w2;
    const float mi = h2f(w0 & 0xffff), di = h2f(w0 >> 16);
    const float mm = h2f(w1 & 0xffff), dm = h2f(w1 >> 16);
    const float mo = h2f(w2 & 0xffff), dd = h2f(w2 >> 16);
    Tok T;
    T.base = th[1] - mm - 7.0f * dm;
    T.dm = dm;
    T.gp = th[2] - th[1] + 2.0f * mm - dm;
    T.b_il = -mi - 15.0f * di;
    T.b_ih = mi;
    T.b_ol = th[0] - mo - 15.0f * dd;
    T.b_oh = th[3] + mo;
    T.kd_i = di - dm;
    T.kd_o = dd - dm;
    return T;
}

// The kernel runs one wave per workgroup.  The LDS operations of a wave execute in
// issue order, so handing data between its lanes through LDS needs no wait at all: only
// wavefront-scope fences, which keep the compiler from moving memory operations across
// the hand-over and emit no instructions.  (A workgroup barrier would wait for every
// global load in flight and stall the prefetch pipeline; draining the LDS counter would
// stall on every outstanding LDS operation.)
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint4 ld16(const uint8_t* p) {
    return *reinterpret_cast<const uint4*>(p);
}

// The correction slots build LDS addresses by OR-ing entry bits into aligned bases, so
// the first members sit at offsets that are multiples of their sizes: tab at 0 (bits
// 10-11 select the class, bit 3 the nibble half), dense at 4096 (a page per 1024 bytes;
// K rows of 64 bytes, V channel rows of 8 bytes), q 256-aligned.
//
// Buffers live only in the phase that needs them share storage, which keeps the wave's
// LDS small enough for more waves per CU: the fixed-point query (qi) is read only
// before the key pass and sits in the table's space; tokc (key pass) shares with the
// value pass's wv and oci, which take turns within a group (wv is read by the matrix-core
// operands before the correction walk clears oci and sums into it), and after the value
// pass with the value corrections on their way to the output lanes.
//
// The correction walks take one token per lane, and the table is token-major: row tg (64
// bytes) holds the four classes at 16-byte slots rotated by bits 1-2 of tg (so that lanes
// reading one class spread over the banks), each slot the two nibble halves.  The key walk
// reads the query heads of a channel in fp16; in the value walk 4 * channel locates both
// the channel's dense dword and its correction.
template <int G>
struct Smem {
    __align__(16) uint8_t tab_[4 * GT * 2 * 8];   // correction table; qi
    __align__(16) uint8_t dense[GRP][PSTR];       // K: token rows of 64 bytes; V: page pairs
                                                  // (vflat)
    __align__(16) uint8_t q_[G * D * 2];          // q (keys)
    __align__(16) uint8_t tw_[cmax(cmax(GT * 16, G * GT * 8), G * D * 4)];
    float pbase[G];
    float m[G], l[G];
    __align__(16) uint8_t head[GRP][CB];          // COO counts of a group's records
    __align__(16) uint8_t sparse[SPL + 80];       // page p's COO bytes at p*SSLOT; + slack for
                                                  // whole-dword reads past a run

    // the dense buffer as bytes (value staging)
    __device__ uint8_t* vflat() { return &dense[0][0]; }
    __device__ const uint8_t* vflat() const { return &dense[0][0]; }
    // query in fixed point (before the key pass)
    __device__ int (&qi())[G][D] { return *reinterpret_cast<int (*)[G][D]>(tab_); }
    // query in fp16, the heads of a channel side by side (key pass)
    __device__ __half (&q16())[D][G] { return *reinterpret_cast<__half (*)[D][G]>(q_); }
    // value corrections of one group, fixed point (value pass)
    __device__ int& oci(int hd, int ch) { return reinterpret_cast<int*>(tw_)[hd * D + ch]; }
    // (two or four heads: heads 2p and 2p + 1 of channel ch packed in one 64-bit sum)
    __device__ unsigned long long& oci2(int hp, int ch) {
        return reinterpret_cast<unsigned long long*>(tw_)[hp * D + ch];
    }
    // base, Delta, Gp of the group's tokens (key pass)
    __device__ float4 (&tokc())[GT] { return *reinterpret_cast<float4 (*)[GT]>(tw_); }
    // value-pass weights of token pairs: 4 features, 4 limbs (value pass)
    __device__ uint4 (&wv())[G][GT / 2] { return *reinterpret_cast<uint4 (*)[G][GT / 2]>(tw_); }
    // value corrections, handed to the output lanes (after the value pass)
    __device__ float (&oc())[G][D] { return *reinterpret_cast<float (*)[G][D]>(tw_); }
};

// A group of consecutive pages of one sequence: wave-uniform record pointers and valid
// slots of its pages, and for each lane those of its own page (lane >> 4).
struct Grp {
    const uint8_t* base[GRP];   // the page's record, or a valid stand-in record when absent
    int nval[GRP];              // valid slots per page (0 when absent or outside the range)
    int npg;
    const uint8_t* mine;        // the record of the lane's page
    int nv;                     // its valid slots
};

// The range's pages, one per lane (lane i: page p_begin + i; a range spans at most 32
// pages, and every lane index read below stays under 64): the byte offset of the page's
// key record from the pool (0, a valid stand-in record, when the page is absent or outside
// the range) and its valid slots (0 then).  Formed once per range, so a group's pages cost
// three lane reads each instead of a block-id check and a 64-bit product.
struct PageLanes {
    uint32_t off_lo, off_hi;
    int nval;
};

__device__ __forceinline__ PageLanes page_lanes(const AttnArgs& a, const int32_t* btab, int p_begin, int p_end,
                                                int L, int h, int lane) {
    const int pi = p_begin + lane;
    const int blk = (pi < p_end) ? btab[pi] : -1;
    const bool ok = blk >= 0 && blk < a.num_blocks;
    const uint64_t off = ok ? (uint64_t)(((int64_t)blk * a.H + h) * 2) * (uint64_t)a.stride : 0u;
    return PageLanes{(uint32_t)off, (uint32_t)(off >> 32), ok ? max(0, min(P, L - pi * P)) : 0};
}

// Group of pages g0 .. g0 + 3 of the range; `rec` is the pool plus `which` record strides.
// Each lane takes its own page's entries from the page table by a lane permute (one LDS
// crossbar read each), so per-page loads need no selection among the group's pointers.
__device__ __forceinline__ Grp make_group(const PageLanes& pl, const uint8_t* rec, int p_begin, int g0, int p_end,
                                          int lane) {
    Grp gr;
    gr.npg = max(0, min(GRP, p_end - g0));
#pragma unroll
    for (int pg = 0; pg < GRP; ++pg) {
        const int li = g0 + pg - p_begin;
        const uint64_t off = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)pl.off_hi, li) << 32) |
                             (uint32_t)__builtin_amdgcn_readlane((int)pl.off_lo, li);
        gr.base[pg] = rec + off;
        gr.nval[pg] = __builtin_amdgcn_readlane(pl.nval, li);
    }
    const int src = (g0 - p_begin + (lane >> 4)) * 4;   // (a lane index below 64: byte address)
    const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)pl.off_lo);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)pl.off_hi);
    gr.mine = rec + (((uint64_t)hi << 32) | lo);
    gr.nv = __builtin_amdgcn_ds_bpermute(src, pl.nval);
    return gr;
}


// Global loads are issued unconditionally, so the compiler never has to merge a loaded
// and a default value (which would make it wait for the load right away and defeat the
// prefetch).  Missing pages read a valid stand-in record whose bytes are never used:
// every consumer masks by the page's valid-slot count.

// One 16-byte chunk of the group's COO counts: lanes 16 p and 16 p + 1 read the two chunks
// of page p (the page's other lanes read the same bytes again).
__device__ __forceinline__ uint4 count_chunk(const Grp& gr, int lane) {
    return ld16(gr.mine + (uint32_t)(lane & 1) * 16u);
}
// Stage the counts read by count_chunk into the head buffer.
template <typename S_>
__device__ __forceinline__ void stage_counts(S_& S, const uint4& hreg, int lane) {
    if ((lane & 15) < 2) *reinterpret_cast<uint4*>(&S.head[lane >> 4][16 * (lane & 1)]) = hreg;
}

// With on-demand sparse pages: the first two entries of the sparse page table of the
// lane's page (lane >> 4), which hold the bytes a staged page can use.
__device__ __forceinline__ int2 page_tab(const Grp& gr, int lane) {
    return *reinterpret_cast<const int2*>(gr.mine + LY.sparse);
}

// The metadata of the lane's token (lane = 16 * page + slot).  Stays in registers until
// the group's token constants are formed.
__device__ __forceinline__ Meta meta_words(const Grp& gr, int lane) {
    const uint32_t* m = reinterpret_cast<const uint32_t*>(gr.mine + LY.meta + 12 * (lane & 15));
    return Meta{m[0], m[1], m[2]};
}

// The COO entries of the lane's token (lane = 16 * page + slot), in stream order: cnt
// entries from byte st of its page's stream, the first c0 of them in chunk 0.  Carried
// between groups packed in one register: st (bits 0-11), c0 (12-19), cnt (20-31).
struct Run {
    int st, c0, cnt;
};
__device__ __forceinline__ uint32_t pack_run(const Run& r) {
    return (uint32_t)r.st | ((uint32_t)r.c0 << 12) | ((uint32_t)r.cnt << 20);
}
__device__ __forceinline__ Run unpack_run(uint32_t x) {
    return Run{(int)(x & 0xfffu), (int)((x >> 12) & 0xffu), (int)(x >> 20)};
}

// Start of each slot's COO bytes in its page, from the group's counts in the head
// buffer.  Returns the COO bytes used by the lane's page (lane >> 4), whether every page
// fits its staging slot, and the lane's own run.
template <int G>
__device__ __forceinline__ int group_layout(Smem<G>& S, const Grp& gr, int lane, bool& fits, Run& run) {
    const int pg = lane >> 4, t = lane & 15;
    const int nv = gr.nv;
    const int c0 = (t < nv) ? (int)S.head[pg][2 * t] : 0;
    const int c1 = (t < nv) ? (int)S.head[pg][2 * t + 1] : 0;
    const int tot = c0 + c1;
    const int incl = row_scan16(tot);
    // a 64-value chunk has at most 64 entries; larger counts are not a valid record
    run.st = incl - tot;
    run.c0 = min(c0, 64);
    run.cnt = max(0, min(run.c0 + min(c1, 64), SPCAP - run.st));
    const int u0 = __builtin_amdgcn_readlane(incl, 15), u1 = __builtin_amdgcn_readlane(incl, 31);
    const int u2 = __builtin_amdgcn_readlane(incl, 47), u3 = __builtin_amdgcn_readlane(incl, 63);
    fits = max(max(u0, u1), max(u2, u3)) <= SSLOT;
    return lane < 16 ? u0 : lane < 32 ? u1 : lane < 48 ? u2 : u3;
}

// Sparse page id from a record table entry (1 + id; 0 = none held), clamped into the
// pool so that a stale or missing entry can only misread, never fault.
__device__ __forceinline__ const uint8_t* sparse_page(const AttnArgs& a, int32_t entry) {
    const int id = entry - 1;
    return a.spool + (int64_t)((id >= 0 && id < a.spages) ? id : 0) * kSparsePage;
}

// The lane's two 16-byte chunks of its page's COO bytes: chunks (lane & 15) and
// (lane & 15) + 16 of page lane >> 4.  Chunks past the page's used bytes re-read chunk 0.
// With on-demand pages the two chunk rows are the record's first two sparse pages.
template <bool PG>
__device__ __forceinline__ void sparse_chunks(const AttnArgs& a, const Grp& gr, int2 tab, int used, int lane,
                                              uint4& r0, uint4& r1) {
    const uint32_t o0 = (uint32_t)(lane & 15) * 16u, o1 = o0 + 256u;
    if constexpr (PG) {
        const uint8_t* p0 = sparse_page(a, tab.x);
        const uint8_t* p1 = sparse_page(a, tab.y);
        r0 = ld16(p0 + ((int)o0 < used ? o0 : 0u));
        r1 = ld16((int)o1 < used ? p1 + o0 : p0);
    } else {
        r0 = ld16(gr.mine + LY.sparse + ((int)o0 < used ? o0 : 0u));
        r1 = ld16(gr.mine + LY.sparse + ((int)o1 < used ? o1 : 0u));
    }
}

// COO byte `off` of the lane's page stream, read from HBM (groups whose pages exceed their
// staging slot).
template <bool PG>
__device__ __forceinline__ uint32_t coo_byte(const AttnArgs& a, const Grp& gr, int off) {
    const uint8_t* r = gr.mine;
    if constexpr (PG) {
        const int32_t entry = reinterpret_cast<const int32_t*>(r + LY.sparse)[off / kSparsePage];
        return sparse_page(a, entry)[off % kSparsePage];
    }
    return r[LY.sparse + off];
}

// Writes the token's correction table: for COO class cls = COO >> 6 (bit 0 outer,
// bit 1 upper side) and nibble n with high bit h, the true value minus the nibble's
// middle reading is x + n*y with (x, y) the float2 at row tg, class slot cls ^ (bits 1-2
// of tg), half h: x = B_cls - base - h*Gp, y = Delta_group - Delta_middle.  Everything is
// scaled by w.
template <int G>
__device__ __forceinline__ void token_table(Smem<G>& S, int tg, const Tok& T, float w) {
    const float x[4] = {T.b_il - T.base, T.b_ol - T.base, T.b_ih - T.base, T.b_oh - T.base};
    const float y[4] = {T.kd_i, T.kd_o, T.kd_i, T.kd_o};
#pragma unroll
    for (int cls = 0; cls < 4; ++cls) {
        float4* row = reinterpret_cast<float4*>(&S.tab_[tg * 64 + ((cls ^ ((tg >> 1) & 3)) << 4)]);
        *row = make_float4(w * x[cls], w * y[cls], w * (x[cls] - T.gp), w * y[cls]);
    }
}

template <typename T, int G>
__device__ __forceinline__ const T& lds_at(const Smem<G>& S, uint32_t off) {
    return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(&S) + off);
}

static_assert(offsetof(Smem<1>, dense) == 4096 && offsetof(Smem<1>, q_) % 256 == 0 &&
              offsetof(Smem<2>, q_) % 256 == 0 && offsetof(Smem<4>, q_) % 256 == 0 &&
              sizeof(Smem<4>::tab_) >= sizeof(int) * 4 * D, "LDS layout the correction addressing relies on");

template <int G>
__device__ __forceinline__ uint32_t off_of(const Smem<G>& S, const void* p) {
    return (uint32_t)(reinterpret_cast<const char*>(p) - reinterpret_cast<const char*>(&S));
}

// ---- correction walks: one token per lane --------------------------------------------
//
// Lane 16*page + slot walks every COO entry of its token, both chunks, as one run of the
// staged stream.  The entries of a dword are decoded together, one byte per entry:
// position bytes (128 + i - c0, whose top bit marks chunk 1), query and dense offsets,
// nibble shifts and table slots.  Each entry then costs one OR per LDS address.  The
// loop runs over the lane's whole dwords of entries (lanes leave it as their runs end),
// and the last 1-3 entries are taken one by one.

__device__ __forceinline__ uint32_t byte_at(uint32_t x, int i) { return (x >> (8 * i)) & 0xffu; }

// base | byte i of x, and byte i of x << s, each one VALU operation with a sub-dword
// operand select (i is a constant after unrolling).
#define OAKEN_SDWA_OR(I)                                                                              \
    asm("v_or_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #I " src1_sel:DWORD" \
        : "=v"(r) : "v"(x), "v"(base))
__device__ __forceinline__ uint32_t or_byte(uint32_t x, uint32_t base, int i) {
    uint32_t r;
    switch (i) {
        case 0: OAKEN_SDWA_OR(0); break;
        case 1: OAKEN_SDWA_OR(1); break;
        case 2: OAKEN_SDWA_OR(2); break;
        default: OAKEN_SDWA_OR(3); break;
    }
    return r;
}
#undef OAKEN_SDWA_OR
#define OAKEN_SDWA_SHL(I)                                                                                  \
    asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_" #I \
        : "=v"(r) : "v"(sh), "v"(x))
__device__ __forceinline__ uint32_t shl_byte(uint32_t x, uint32_t sh, int i) {
    uint32_t r;
    switch (i) {
        case 0: OAKEN_SDWA_SHL(0); break;
        case 1: OAKEN_SDWA_SHL(1); break;
        case 2: OAKEN_SDWA_SHL(2); break;
        default: OAKEN_SDWA_SHL(3); break;
    }
    return r;
}
#undef OAKEN_SDWA_SHL

// Query-head count as a shift (G = 1, 2, 4).
template <int G>
constexpr int log2g() { return G == 1 ? 0 : G == 2 ? 1 : 2; }

// One fp16 query head of a channel's heads (loaded together) into a float.
template <int G>
__device__ __forceinline__ float q_head(const uint2& qv, int hd) {
    const uint32_t w = hd < 2 ? qv.x : qv.y;
    return __half2float(__ushort_as_half((uint16_t)((hd & 1) ? (w >> 16) : (w & 0xffffu))));
}

// The G fp16 query heads of the channel at byte offset qa (G * 2 bytes).
template <int G>
__device__ __forceinline__ uint2 q_heads(const Smem<G>& S, uint32_t qa) {
    if constexpr (G == 4) return lds_at<uint2>(S, qa);
    else if constexpr (G == 2) return make_uint2(lds_at<uint32_t>(S, qa), 0u);
    else return make_uint2((uint32_t)lds_at<uint16_t>(S, qa), 0u);
}

// Scores: each entry adds q_j * (true value - middle reading) to its token's score, for
// each of the G query heads; corr receives the lane's token's sums (before the scale).
template <int G, bool PG>
__device__ __forceinline__ void key_corrections(Smem<G>& S, const AttnArgs& a, const Run& r, bool staged,
                                                const Grp& gr, int lane, float (&corr)[G]) {
    constexpr int QS = 1 + log2g<G>();                            // log2 of the query bytes per channel
    const int pg = lane >> 4, t = lane & 15;
    const uint32_t tbo = (uint32_t)lane * 64u;                    // the token's table row
    const uint32_t swz = (uint32_t)((lane >> 1) & 3) * 0x10101010u;
    const uint32_t qb = off_of(S, &S.q16()[0][0]);                // 256-aligned
    const uint32_t drow = off_of(S, &S.dense[pg][t * 64]);        // 64-aligned
#pragma unroll
    for (int hd = 0; hd < G; ++hd) corr[hd] = 0.0f;
    // one entry: query offset qo (channel << QS), dense offset byte dof (dword of the
    // channel within the token row), nibble shift ns, table slot byte ct
    auto entry = [&](uint32_t qo, uint32_t dof, uint32_t ns, uint32_t ct) {
        const uint32_t dw = lds_at<uint32_t>(S, drow | dof);
        const uint2 qv = q_heads<G>(S, qb + qo);
        const uint32_t n = __builtin_amdgcn_ubfe(dw, ns, 4);
        const float2 kv = lds_at<float2>(S, (tbo | ct) | (n & 8u));
        const float delta = fmaf((float)n, kv.y, kv.x);
#pragma unroll
        for (int hd = 0; hd < G; ++hd) corr[hd] = fmaf(q_head<G>(qv, hd), delta, corr[hd]);
    };
    if (staged) {
        const int pos = pg * SSLOT + r.st;
        const uint32_t* w = reinterpret_cast<const uint32_t*>(&S.sparse[pos & ~3]);
        const uint32_t sh = pos & 3;
        uint32_t cur = w[0], nxt = w[1];
        // position bytes 64 + i - c0 of entries i..i+3: bit 6 marks chunk 1 (a chunk holds at
        // most 64 entries, so the used bytes stay below 128)
        const uint32_t pc0 = 0x03020100u + (uint32_t)(64 - r.c0) * 0x01010101u;
        // per dword: channels (7 bits, chunk on top), dense offsets, raw entries (nibble
        // shifts), table slots
        auto decode = [&](int kk, uint32_t& ch4, uint32_t& do4, uint32_t& ent, uint32_t& ct4) {
            ent = __builtin_amdgcn_alignbyte(nxt, cur, sh);
            const uint32_t pcb = pc0 + (uint32_t)kk * 0x01010101u;
            ch4 = (ent & 0x3f3f3f3fu) | (pcb & 0xc0c0c0c0u);        // channel
            do4 = (ch4 >> 1) & 0x3c3c3c3cu;                         // (channel / 8) * 4
            ct4 = ((ent >> 2) & 0x30303030u) ^ swz;
        };
        const int full = r.cnt & ~3;
        for (int kk = 0; kk < full; kk += 4) {
            uint32_t ch4, do4, ent, ct4;
            decode(kk, ch4, do4, ent, ct4);
            // the next block's pair of dwords, read whole (no register shuffle between blocks)
            cur = w[(kk >> 2) + 1];
            nxt = w[(kk >> 2) + 2];
            // phases kept apart so that a dword's reads issue together
            uint32_t dw[4];
            uint2 qv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                dw[i] = lds_at<uint32_t>(S, or_byte(do4, drow, i));
                qv[i] = q_heads<G>(S, qb + shl_byte(ch4, (uint32_t)QS, i));
            }
            __builtin_amdgcn_sched_barrier(0);
            uint32_t n[4];
            float2 kv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                n[i] = __builtin_amdgcn_ubfe(dw[i], shl_byte(ent, 2u, i), 4);
                kv[i] = lds_at<float2>(S, or_byte(ct4, tbo, i) | (n[i] & 8u));
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float delta = fmaf((float)n[i], kv[i].y, kv[i].x);
#pragma unroll
                for (int hd = 0; hd < G; ++hd) corr[hd] = fmaf(q_head<G>(qv[i], hd), delta, corr[hd]);
            }
        }
        if (full < r.cnt) {
            uint32_t ch4, do4, ent, ct4;
            decode(full, ch4, do4, ent, ct4);
            entry(byte_at(ch4, 0) << QS, byte_at(do4, 0), byte_at(ent, 0) << 2, byte_at(ct4, 0));
            if (full + 1 < r.cnt) entry(byte_at(ch4, 1) << QS, byte_at(do4, 1), byte_at(ent, 1) << 2, byte_at(ct4, 1));
            if (full + 2 < r.cnt) entry(byte_at(ch4, 2) << QS, byte_at(do4, 2), byte_at(ent, 2) << 2, byte_at(ct4, 2));
        }
    } else {
        for (int kk = 0; kk < r.cnt; ++kk) {
            const uint32_t b = coo_byte<PG>(a, gr, r.st + kk);
            const uint32_t ch = (b & 63u) | (kk >= r.c0 ? 64u : 0u);
            entry(ch << QS, (ch >> 3) * 4u, (ch & 7u) * 4u, ((b >> 2) & 0x30u) ^ (swz & 0xffu));
        }
    }
}

// Values: each entry adds p_t * (true value - middle reading) to its channel, once per
// query head, in the group's fixed point.  With one head the table already carries p_t.
template <int G, bool PG>
__device__ __forceinline__ void value_corrections(Smem<G>& S, const AttnArgs& a, const float* sc, int cap,
                                                  const Run& r, bool staged, const Grp& gr, int tok0, int lane) {
    const int pg = lane >> 4, t = lane & 15;
    const uint32_t tbo = (uint32_t)lane * 64u;
    const uint32_t swz = (uint32_t)((lane >> 1) & 3) * 0x10101010u;
    // the token's dwords: + 8 * channel
    const uint32_t dcol = off_of(S, S.vflat() + vpos(pg) + (t >> 3) * 4);
    const uint32_t nsh = (uint32_t)(t & 7) * 4u;
    const uint32_t occ = off_of(S, &S.oci(0, 0));                     // + 4 * channel (+ 4 D * head)
    float pt[G];
    const int nv = gr.nv;
#pragma unroll
    for (int hd = 0; hd < G; ++hd) pt[hd] = (G > 1 && t < nv) ? sc[hd * cap + tok0 + lane] : 1.0f;
    auto add = [&](uint32_t x, float delta) {
        if constexpr (G == 1) {
            atomicAdd(&const_cast<int&>(lds_at<int>(S, occ + x)), (int)delta);
        } else {
            // two heads per 64-bit add: (v1 + borrow) * 2^32 + v0 sums exactly to
            // S1 * 2^32 + S0 while each head's sum stays within 32 bits
            const uint32_t o8 = occ + 2 * x;
#pragma unroll
            for (int hp = 0; hp < G / 2; ++hp) {
                const int v0 = (int)(pt[2 * hp] * delta), v1 = (int)(pt[2 * hp + 1] * delta);
                const uint64_t pk = ((uint64_t)(uint32_t)(v1 + (v0 >> 31)) << 32) | (uint32_t)v0;
                atomicAdd(&const_cast<unsigned long long&>(lds_at<unsigned long long>(S, o8 + hp * D * 8)),
                          (unsigned long long)pk);
            }
        }
    };
    // one entry: channel offset x = 4 * channel, table slot byte ct
    auto entry = [&](uint32_t x, uint32_t ct) {
        const uint32_t dw = lds_at<uint32_t>(S, dcol + 2 * x);
        const uint32_t n = __builtin_amdgcn_ubfe(dw, nsh, 4);
        const float2 kv = lds_at<float2>(S, (tbo | ct) | (n & 8u));
        add(x, fmaf((float)n, kv.y, kv.x));
    };
    if (staged) {
        const int pos = pg * SSLOT + r.st;
        const uint32_t* w = reinterpret_cast<const uint32_t*>(&S.sparse[pos & ~3]);
        const uint32_t sh = pos & 3;
        uint32_t cur = w[0], nxt = w[1];
        // position bytes 64 + i - c0 of entries i..i+3: bit 6 marks chunk 1 (a chunk holds at
        // most 64 entries, so the used bytes stay below 128)
        const uint32_t pc0 = 0x03020100u + (uint32_t)(64 - r.c0) * 0x01010101u;
        auto decode = [&](int kk, uint32_t& ch4, uint32_t& ct4) {
            const uint32_t ent = __builtin_amdgcn_alignbyte(nxt, cur, sh);
            const uint32_t pcb = pc0 + (uint32_t)kk * 0x01010101u;
            ch4 = (ent & 0x3f3f3f3fu) | (pcb & 0xc0c0c0c0u);      // channel per byte
            ct4 = ((ent >> 2) & 0x30303030u) ^ swz;
        };
        const int full = r.cnt & ~3;
        for (int kk = 0; kk < full; kk += 4) {
            uint32_t ch4, ct4;
            decode(kk, ch4, ct4);
            // the next block's pair of dwords, read whole (no register shuffle between blocks)
            cur = w[(kk >> 2) + 1];
            nxt = w[(kk >> 2) + 2];
            uint32_t x[4], dw[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x[i] = shl_byte(ch4, 2u, i);
                dw[i] = lds_at<uint32_t>(S, dcol + 2 * x[i]);
            }
            __builtin_amdgcn_sched_barrier(0);
            uint32_t n[4];
            float2 kv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                n[i] = __builtin_amdgcn_ubfe(dw[i], nsh, 4);
                kv[i] = lds_at<float2>(S, or_byte(ct4, tbo, i) | (n[i] & 8u));
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < 4; ++i) add(x[i], fmaf((float)n[i], kv[i].y, kv[i].x));
        }
        if (full < r.cnt) {
            uint32_t ch4, ct4;
            decode(full, ch4, ct4);
            entry(byte_at(ch4, 0) << 2, byte_at(ct4, 0));
            if (full + 1 < r.cnt) entry(byte_at(ch4, 1) << 2, byte_at(ct4, 1));
            if (full + 2 < r.cnt) entry(byte_at(ch4, 2) << 2, byte_at(ct4, 2));
        }
    } else {
        for (int kk = 0; kk < r.cnt; ++kk) {
            const uint32_t b = coo_byte<PG>(a, gr, r.st + kk);
            const uint32_t ch = (b & 63u) | (kk >= r.c0 ? 64u : 0u);
            entry(ch * 4u, ((b >> 2) & 0x30u) ^ (swz & 0xffu));
        }
    }
}

// Three waves per SIMD (168 registers), except four heads over on-demand sparse pages, which
// would spill there and take what they need (two waves per SIMD).
template <int G, bool PG>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(G == 4 && PG ? 1 : 3))) void attn_mfma_kernel(AttnArgs a) {
    constexpr int NRS = (G + 1) / 2;        // key-pass MFMA row sets (8 rows per head)
    __shared__ Smem<G> S;
    extern __shared__ float sc[];           // [G][cap]: scores, then probabilities

    const int lane = threadIdx.x;
    const AttnTile tile = attn_tile(a);
    const int split = tile.split, h = tile.h, s = tile.s;
    const int qh0 = h * (a.Hq / a.H) + tile.part * G;   // the workgroup's first query head
    const int L = max(0, min(a.seq_lens[s], min(a.max_seq_len, a.max_blocks * P)));
    const int n_pages = (L + P - 1) / P;
    // a sliding window hides keys before lo; the ranges start at its first page
    const int lo = (a.window > 0 && L > a.window) ? L - a.window : 0;
    const int p_begin = lo / P + split * a.pages_per_split;
    const int p_end = min(n_pages, p_begin + a.pages_per_split);
    const int cap = a.pages_per_split * P;
    const int n_tok = max(0, min(L, p_end * P) - p_begin * P);
    // a range past the end of a shorter sequence of the batch: an empty partial (l = 0,
    // which the combine skips) and nothing else
    if (n_tok <= 0 && a.n_splits > 1) {
        if (lane < G) {
            float* pp = a.partial + (((int64_t)s * a.Hq + qh0 + lane) * a.n_splits + split) * (D + 2);
            pp[D] = -INFINITY;
            pp[D + 1] = 0.0f;
        }
        return;
    }
    const int32_t* btab = a.block_table + (int64_t)s * a.max_blocks;
    constexpr bool paged = PG;   // on-demand sparse pages
    const PageLanes pl = page_lanes(a, btab, p_begin, p_end, L, h, lane);
    const uint8_t* const krec = a.pool;
    const uint8_t* const vrec = a.pool + a.stride;

    float tk[4], tv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        tk[i] = fin(a.thr[(h * 2 + 0) * 4 + i]);
        tv[i] = fin(a.thr[(h * 2 + 1) * 4 + i]);
    }

    // the first key group's counts and metadata are needed before anything else
    Grp gc = make_group(pl, krec, p_begin, p_begin, p_end, lane);
    uint4 hreg = count_chunk(gc, lane);
    int2 tab_c = paged ? page_tab(gc, lane) : int2{0, 0};   // (on-demand sparse pages)
    Meta mreg = meta_words(gc, lane);

    // ---- query in fp32 and in fixed point -----------------------------------------
    float ssum[G], sfix[G];
#pragma unroll
    for (int hd = 0; hd < G; ++hd) {
        const uint16_t* qp = a.q + ((int64_t)s * a.Hq + qh0 + hd) * D;
        const float x0 = h2f(qp[lane]), x1 = h2f(qp[lane + 64]);
        S.q16()[lane][hd] = __ushort_as_half(qp[lane]);
        S.q16()[lane + 64][hd] = __ushort_as_half(qp[lane + 64]);
        const float mx = wave_max_nonneg(fmaxf(fabsf(x0), fabsf(x1)));
        const float sum = wave_sum(x0 + x1);
        const int sh = fix_shift(mx);
        S.qi()[hd][lane] = (int)rintf(ldexpf(x0, sh));
        S.qi()[hd][lane + 64] = (int)rintf(ldexpf(x1, sh));
        // score = scale * (base * sum(q) + (Delta * U + Gp * H) * 2^-(shift + 7))
        ssum[hd] = a.scale * sum;
        sfix[hd] = ldexpf(a.scale, -(sh + 7));
    }
    stage_counts(S, hreg, lane);
    wave_sync();

    // Key-pass A operand: row = 8*(head%2) + 4*type + limb, type 0 -> sum q u, 1 -> sum q h.
    // MFMA f takes feature f of the lane's 16 dense bytes: its byte (4m + b) of k-group g4
    // pairs with feature f of dense byte 16*g4 + 4*m + b.  The raw-byte operand is then the
    // loaded register itself and the others one AND per dword.
    // Each lane first encodes the eight limb words of dense byte `lane` (channels 2 lane and
    // 2 lane + 1) for each head of the row set into LDS (the dense staging area, unused until
    // the key loop); a lane then gathers limb r of four bytes with three byte permutes.
    v4i afk[NRS][4];
    {
        // (a copy of the lane id the compiler cannot see through, so that no address formed
        // here is kept alive for reuse in the loops)
        int ln;
        asm volatile("v_mov_b32 %0, %1" : "=v"(ln) : "v"(lane));
        const int row = ln & 15, g4 = ln >> 4, type = (row >> 2) & 1, r = row & 3;
        uint32_t* E = reinterpret_cast<uint32_t*>(&S.dense[0][0]);   // [2 heads][2 types][4 features][64 bytes]
        const uint32_t sel = (uint32_t)r | ((uint32_t)(r + 4) << 8);
#pragma unroll
        for (int rs = 0; rs < NRS; ++rs) {
#pragma unroll
            for (int hl = 0; hl < 2; ++hl) {
                if (rs * 2 + hl < G) {
                    const int2 qq = *reinterpret_cast<const int2*>(&S.qi()[rs * 2 + hl][2 * ln]);
                    const int qe = qq.x, qo = qq.y;
                    uint32_t* e = E + hl * 512 + ln;
                    // the weights of (raw byte, low nibble, bits 7|3, bit 3) for sum q u ...
                    e[0 * 64] = enc(8 * qo);
                    e[1 * 64] = enc(128 * qe - 8 * qo);
                    e[2 * 64] = enc(-16 * qo);
                    e[3 * 64] = enc(16 * qo);
                    // ... and for sum q h
                    e[4 * 64] = 0u;
                    e[5 * 64] = 0u;
                    e[6 * 64] = enc(-qo);
                    e[7 * 64] = enc(16 * qe + qo);
                }
            }
            wave_sync();
            const bool live = rs * 2 + (row >> 3) < G;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
#pragma unroll
                for (int f = 0; f < 4; ++f) {
                    uint32_t x = 0;
                    if (live) {
                        const uint4 w = *reinterpret_cast<const uint4*>(
                            &E[(row >> 3) * 512 + (type * 4 + f) * 64 + g4 * 16 + m * 4]);
                        const uint32_t t01 = __builtin_amdgcn_perm(w.y, w.x, sel);
                        const uint32_t t23 = __builtin_amdgcn_perm(w.w, w.z, sel);
                        x = __builtin_amdgcn_perm(t23, t01, 0x05040100u);
                    }
                    afk[rs][f][m] = (int)x;
                }
            }
            if (rs + 1 < NRS) wave_sync();   // (the next row set's words replace these)
        }
    }

    // ---- pass 1: keys -------------------------------------------------------------
    uint4 dreg[GRP], sreg0, sreg1;
    const uint32_t koff = (uint32_t)LY.dense + (uint32_t)((lane & 15) * 64 + (lane >> 4) * 16);
    const uint32_t voff = (uint32_t)LY.dense + (uint32_t)lane * 16u;
    const uint32_t stg = (uint32_t)((lane >> 4) * SSLOT + (lane & 15) * 16);   // LDS staging slot
    // (a staged page fits its slot, so its second chunk row is needed only within it)
    const bool stg1_in = 256 + (lane & 15) * 16 < SSLOT;
    bool fits_c, fits_n;
    uint32_t run_c, run_n;   // (one head) the lane's COO run in the current and the next group
    {
        Run r;
        const int used = group_layout(S, gc, lane, fits_c, r);
        run_c = pack_run(r);
        wave_sync();
#pragma unroll
        for (int pg = 0; pg < GRP; ++pg) dreg[pg] = ld16(gc.base[pg] + koff);
        // (one head: issued in the loop's own order, dense bytes first, so that the wait
        // counts at the loop head cover only what the first group needs first; with more
        // heads the fixed order costs register spills)
        if constexpr (G == 1) __builtin_amdgcn_sched_barrier(0);
        sparse_chunks<PG>(a, gc, tab_c, used, lane, sreg0, sreg1);
        if constexpr (G == 1) __builtin_amdgcn_sched_barrier(0);
    }
    Grp gn = make_group(pl, krec, p_begin, p_begin + GRP, p_end, lane);
    hreg = count_chunk(gn, lane);
    int2 tab_n = paged ? page_tab(gn, lane) : int2{0, 0};
    for (int g0 = p_begin; g0 < p_end; g0 += GRP) {
        const int tok0 = (g0 - p_begin) * P;
        const bool staged = fits_c;
        float dot1 = 0.0f;     // one head: the lane's token's dense score
        bool valid1 = false;
        // dense part on the matrix cores: one accumulator per page and the pages' MFMAs
        // interleaved, so that no MFMA waits on the one before it; stage the group in LDS
        {
            v4i acc[GRP][NRS];
#pragma unroll
            for (int pg = 0; pg < GRP; ++pg)
#pragma unroll
                for (int rs = 0; rs < NRS; ++rs) acc[pg][rs] = v4i{0, 0, 0, 0};
#pragma unroll
            for (int f = 0; f < 4; ++f) {
#pragma unroll
                for (int pg = 0; pg < GRP; ++pg) {
                    const v4i B = feature_of(dreg[pg], f);
#pragma unroll
                    for (int rs = 0; rs < NRS; ++rs) acc[pg][rs] = mfma(afk[rs][f], B, acc[pg][rs]);
                }
            }
#pragma unroll
            for (int pg = 0; pg < GRP; ++pg)
                *reinterpret_cast<uint4*>(&S.dense[pg][(lane & 15) * 64 + (lane >> 4) * 16]) = dreg[pg];
            // the next group's dense bytes go out as soon as these are consumed
#pragma unroll
            for (int pg = 0; pg < GRP; ++pg) dreg[pg] = ld16(gn.base[pg] + koff);
            // token constants of the group (lane = token) and the key correction tables,
            // while the MFMAs drain
            {
                const Tok T = token_consts(mreg, tk);
                S.tokc()[lane] = make_float4(T.base, T.dm, T.gp, 0.0f);
                token_table(S, lane, T, 1.0f);
            }
            wave_sync();
            // Lane (t + 16*grp4) holds rows 4*grp4 .. 4*grp4+3 of column t of each page's
            // tile: the U (grp4 even) or H (grp4 odd) limbs of head rs*2 + grp4/2.
            const int t = lane & 15, grp4 = lane >> 4;
            if constexpr (G == 1) {
                // rows 8-15 are zero (no second head): two 16-lane swaps and two 32-lane swaps
                // give lane group p the U and H sums of page p (its lane is its token), so
                // every lane forms one score
                static_assert(GRP == 4, "four pages, one per lane group");
                float v[GRP];
#pragma unroll
                for (int pg = 0; pg < GRP; ++pg) v[pg] = limbs(acc[pg][0]);
                const auto s01 = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, v[0]),
                                                                  __builtin_bit_cast(int, v[1]), false, false);
                const auto s23 = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, v[2]),
                                                                  __builtin_bit_cast(int, v[3]), false, false);
                const float u = __builtin_bit_cast(float, (int)__builtin_amdgcn_permlane32_swap(s01[0], s23[0], false, false)[0]);
                const float o = __builtin_bit_cast(float, (int)__builtin_amdgcn_permlane32_swap(s01[1], s23[1], false, false)[0]);
                const float4 tc = S.tokc()[lane];
                // (the score is stored once, after the correction walk has added to it)
                valid1 = t < gc.nv && (g0 + grp4) * P + t >= lo;
                dot1 = fmaf(tc.x, ssum[0], fmaf(tc.y, u, tc.z * o) * sfix[0]);
            } else {
                // (per page: the paired form of the one-head case spills registers here)
                // rows 1 and 3 reach rows 0 and 2 by a row swap
                const bool hi = (grp4 >> 1) != 0;
#pragma unroll
                for (int pg = 0; pg < GRP; ++pg) {
                    const float4 tc = S.tokc()[pg * P + t];
                    const bool valid = t < gc.nval[pg] && (g0 + pg) * P + t >= lo;
#pragma unroll
                    for (int rs = 0; rs < NRS; ++rs) {
                        const float v = limbs(acc[pg][rs]);
                        const int vb = __builtin_bit_cast(int, v);
                        const float o = __builtin_bit_cast(float, (int)__builtin_amdgcn_permlane16_swap(vb, vb, false, false)[1]);
                        const int hd = rs * 2 + (hi ? 1 : 0);
                        const float s1 = hi ? ssum[min(rs * 2 + 1, G - 1)] : ssum[rs * 2];
                        const float s2 = hi ? sfix[min(rs * 2 + 1, G - 1)] : sfix[rs * 2];
                        const float dot = fmaf(tc.x, s1, fmaf(tc.y, v, tc.z * o) * s2);
                        if ((grp4 & 1) == 0 && hd < G && pg < gc.npg)
                            sc[hd * cap + tok0 + pg * P + t] = valid ? dot : -INFINITY;
                    }
                }
            }
        }
        if (staged) {
            *reinterpret_cast<uint4*>(&S.sparse[stg]) = sreg0;
            if (stg1_in) *reinterpret_cast<uint4*>(&S.sparse[stg + 256]) = sreg1;
        }
        wave_sync();
        // next group: heads -> layout -> issue its sparse bytes and the heads after it.
        // Also past the range's last group (stand-in records without valid slots): every
        // path through the loop then has the same loads in flight, so the compiler's wait
        // counts stay exact instead of draining the whole prefetch at the loop's edges.
        Grp gnn;
        int2 tab_nn = tab_n;
        {
            // (the metadata first: the next group needs it before its sparse bytes)
            mreg = meta_words(gn, lane);
            stage_counts(S, hreg, lane);
            wave_sync();
            Run r;
            const int used = group_layout(S, gn, lane, fits_n, r);
            run_n = pack_run(r);
            wave_sync();
            sparse_chunks<PG>(a, gn, tab_n, used, lane, sreg0, sreg1);
            gnn = make_group(pl, krec, p_begin, g0 + 2 * GRP, p_end, lane);
            hreg = count_chunk(gnn, lane);
            if constexpr (PG) tab_nn = page_tab(gnn, lane);
        }
        wave_sync();
        // sparse part
        {
            float corr[G];
            key_corrections<G, PG>(S, a, unpack_run(run_c), staged, gc, lane, corr);
            if constexpr (G == 1) {
                if ((lane >> 4) < gc.npg) sc[tok0 + lane] = valid1 ? dot1 + a.scale * corr[0] : -INFINITY;
            } else if ((lane & 15) < gc.nv) {
#pragma unroll
                for (int hd = 0; hd < G; ++hd) sc[hd * cap + tok0 + lane] += a.scale * corr[hd];
            }
        }
        wave_sync();
        gc = gn;
        gn = gnn;
        tab_n = tab_nn;
        fits_c = fits_n;
        run_c = run_n;
    }

    // the first value group's heads go out before the softmax
    gc = make_group(pl, vrec, p_begin, p_begin, p_end, lane);
    hreg = count_chunk(gc, lane);
    if constexpr (PG) tab_c = page_tab(gc, lane);
    mreg = meta_words(gc, lane);

    // ---- softmax over the range ----------------------------------------------------
#pragma unroll
    for (int hd = 0; hd < G; ++hd) {
        float mx = -INFINITY;
        for (int i = lane; i < n_tok; i += 64) mx = fmaxf(mx, sc[hd * cap + i]);
        mx = wave_max(mx);
        float sum = 0.0f;
        for (int i = lane; i < n_tok; i += 64) {
            const float pr = (mx == -INFINITY) ? 0.0f : __expf(sc[hd * cap + i] - mx);
            sc[hd * cap + i] = pr;
            sum += pr;
        }
        sum = wave_sum(sum);
        if (lane == 0) {
            S.m[hd] = mx;
            S.l[hd] = sum;
        }
    }
    stage_counts(S, hreg, lane);
    wave_sync();

    // ---- pass 2: values ------------------------------------------------------------
    // Output lane (head hq, dim 16*nt + (lane&15)) for several heads.  With one head the
    // sums of tiles nt = 4*hf + hq (hf = 0, 1) are gathered into row group hq first, so that
    // every lane converts two tiles.
    const int hq = lane >> 4;
    constexpr int NO = G == 1 ? 2 : 8;
    float oacc[NO];
#pragma unroll
    for (int nt = 0; nt < NO; ++nt) oacc[nt] = 0.0f;
    float pb[G];
    float ocr[G][2];   // value corrections of channels lane and lane + 64
#pragma unroll
    for (int hd = 0; hd < G; ++hd) pb[hd] = ocr[hd][0] = ocr[hd][1] = 0.0f;
    {
        Run r;
        const int used = group_layout(S, gc, lane, fits_c, r);
        run_c = pack_run(r);
        wave_sync();
#pragma unroll
        for (int pg = 0; pg < GRP; ++pg) dreg[pg] = ld16(gc.base[pg] + voff);
        if constexpr (G == 1) __builtin_amdgcn_sched_barrier(0);   // (as for the keys)
        sparse_chunks<PG>(a, gc, tab_c, used, lane, sreg0, sreg1);
        if constexpr (G == 1) __builtin_amdgcn_sched_barrier(0);
    }
    gn = make_group(pl, vrec, p_begin, p_begin + GRP, p_end, lane);
    hreg = count_chunk(gn, lane);
    if constexpr (PG) tab_n = page_tab(gn, lane);
    for (int g0 = p_begin; g0 < p_end; g0 += GRP) {
        const int tok0 = (g0 - p_begin) * P;
        const bool staged = fits_c;
#pragma unroll
        for (int pg = 0; pg < GRP; ++pg) *reinterpret_cast<uint4*>(S.vflat() + vpos(pg) + lane * 16) = dreg[pg];
        // the next group's dense bytes go out as soon as these are staged
#pragma unroll
        for (int pg = 0; pg < GRP; ++pg) dreg[pg] = ld16(gn.base[pg] + voff);
        if (staged) {
            *reinterpret_cast<uint4*>(&S.sparse[stg]) = sreg0;
            if (stg1_in) *reinterpret_cast<uint4*>(&S.sparse[stg + 256]) = sreg1;
        }
        // fixed-point coefficients p*Delta, p*Gp of the group's tokens (lane = token), one
        // shift per head; correction tables (scaled by p when one head reads them)
        int vsh;   // one fixed-point shift for every head of the group
        int fsh;
        {
            const int t = lane & 15;
            const int nv = gc.nv;
            const bool vt = t < nv;
            const Tok T = token_consts(mreg, tv);
            float p0 = 0.0f, cx[G], gx[G], mx = 0.0f;
#pragma unroll
            for (int hd = 0; hd < G; ++hd) {
                const float p = vt ? sc[hd * cap + tok0 + lane] : 0.0f;
                if (hd == 0) p0 = p;
                cx[hd] = vt ? p * T.dm : 0.0f;
                gx[hd] = vt ? p * T.gp : 0.0f;
                if (vt) pb[hd] = fmaf(p, T.base, pb[hd]);
                mx = fmaxf(mx, fmaxf(fabsf(cx[hd]), fabsf(gx[hd])));
            }
            // (a head whose weights are far below the group's largest keeps fewer bits, but
            // its group then adds little next to its own range total, which is at least 1)
            vsh = fix_shift(wave_max_nonneg(mx));
#pragma unroll
            for (int hd = 0; hd < G; ++hd) {
                // Weights of token pair lane/2 (even lane: its own C, G and the odd
                // partner's): 128 (C_e u_e + C_o u_o + G_e h_e + G_o h_o) over the features
                // (raw byte, low nibble, bits 7|3, bit 3) of the nibble byte, as 4 limbs each.
                const int ce = (int)rintf(ldexpf(cx[hd], vsh)), ge = (int)rintf(ldexpf(gx[hd], vsh));
                const int co = __builtin_amdgcn_update_dpp(0, ce, 0x101, 0xf, 0xf, false);   // row_shl:1
                const int go = __builtin_amdgcn_update_dpp(0, ge, 0x101, 0xf, 0xf, false);
                if ((lane & 1) == 0)
                    S.wv()[hd][lane >> 1] = make_uint4(enc(8 * co), enc(128 * ce - 8 * co), enc(-(go + 16 * co)),
                                                     enc(16 * ge + go + 16 * co));
            }
            // Value corrections accumulate as integers (LDS float atomics are slow): the
            // table is scaled by 2^fsh, chosen so that 64 tokens' largest corrections
            // stay below 2^30 in magnitude.
            const float w = vt ? (G == 1 ? p0 : 1.0f) : 0.0f;
            // (invalid tokens' metadata is arbitrary: they contribute 0, never NaN)
            const float bound = vt ? w * (fmaxf(fmaxf(fabsf(T.b_il - T.base), fabsf(T.b_ol - T.base)),
                                                fmaxf(fabsf(T.b_ih - T.base), fabsf(T.b_oh - T.base))) +
                                          15.0f * fmaxf(fabsf(T.kd_i), fabsf(T.kd_o)) + fabsf(T.gp))
                                   : 0.0f;
            const float gb = wave_max_nonneg(bound);
            int ge = 0;
            if (gb > 0.0f) frexpf(gb, &ge);
            fsh = gb > 0.0f ? 24 - ge : 0;
            const float ws = ldexpf(w, fsh);
            token_table(S, lane, T, ws);
        }
        wave_sync();
        // next group: heads -> layout -> issue its sparse bytes and the heads after it.
        // Also past the range's last group (stand-in records without valid slots): every
        // path through the loop then has the same loads in flight, so the compiler's wait
        // counts stay exact instead of draining the whole prefetch at the loop's edges.
        Grp gnn;
        int2 tab_nn = tab_n;
        {
            // (the metadata first: the next group needs it before its sparse bytes)
            mreg = meta_words(gn, lane);
            stage_counts(S, hreg, lane);
            wave_sync();
            Run r;
            const int used = group_layout(S, gn, lane, fits_n, r);
            run_n = pack_run(r);
            wave_sync();
            sparse_chunks<PG>(a, gn, tab_n, used, lane, sreg0, sreg1);
            gnn = make_group(pl, vrec, p_begin, g0 + 2 * GRP, p_end, lane);
            hreg = count_chunk(gnn, lane);
            if constexpr (PG) tab_nn = page_tab(gnn, lane);
        }
        wave_sync();
        v4i gacc[8];
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) gacc[nt] = v4i{0, 0, 0, 0};
        {
            // A operand of lane (row = 4*head + limb r, k-group g4): for each feature f the
            // limb-r bytes of token pairs 4*g4 + 0..3 of page pair pq (a byte transpose).
            // MFMA 0 takes features 0 and 1, MFMA 1 features 2 and 3, each of the pages
            // g4/2 (pair 0) and g4/2 + 2 (pair 1): A and B registers line up as (pair 0,
            // pair 1) of the first feature, then of the second.
            const int row = lane & 15, hdr = row >> 2, g4 = lane >> 4, r = row & 3;
            v4i av[2] = {v4i{0, 0, 0, 0}, v4i{0, 0, 0, 0}};
            if (hdr < G) {
                const uint32_t sel = (uint32_t)r | ((uint32_t)(r + 4) << 8);
                auto col = [&](uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3) {
                    const uint32_t t01 = __builtin_amdgcn_perm(a1, a0, sel);
                    const uint32_t t23 = __builtin_amdgcn_perm(a3, a2, sel);
                    return (int)__builtin_amdgcn_perm(t23, t01, 0x05040100u);
                };
#pragma unroll
                for (int pq = 0; pq < 2; ++pq) {
                    const uint4* wp = &S.wv()[hdr][pq * 16 + g4 * 4];
                    const uint4 w0 = wp[0], w1 = wp[1], w2 = wp[2], w3 = wp[3];
                    av[pq][0] = col(w0.x, w1.x, w2.x, w3.x);
                    av[pq][1] = col(w0.y, w1.y, w2.y, w3.y);
                    av[pq][2] = col(w0.z, w1.z, w2.z, w3.z);
                    av[pq][3] = col(w0.w, w1.w, w2.w, w3.w);
                }
            }
            const v4i A0 = v4i{av[0][0], av[1][0], av[0][1], av[1][1]};
            const v4i A1 = v4i{av[0][2], av[1][2], av[0][3], av[1][3]};
            const uint8_t* dsrc = S.vflat() + vpos(g4 >> 1) + (g4 & 1) * 4;
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) {
                const int j = nt * 16 + (lane & 15);
                const uint2 dd = make_uint2(*reinterpret_cast<const uint32_t*>(dsrc + j * 8),
                                            *reinterpret_cast<const uint32_t*>(dsrc + 1024 + j * 8));
                const v4i B0 = v4i{(int)dd.x, (int)dd.y, (int)(dd.x & 0x0f0f0f0fu), (int)(dd.y & 0x0f0f0f0fu)};
                const v4i B1 = v4i{(int)(dd.x & 0x88888888u), (int)(dd.y & 0x88888888u), (int)(dd.x & 0x08080808u),
                                   (int)(dd.y & 0x08080808u)};
                gacc[nt] = mfma(A0, B0, gacc[nt]);
                gacc[nt] = mfma(A1, B1, gacc[nt]);
            }
        }
        // the dense sums leave the accumulators before the correction walk, which then has
        // their registers
        if constexpr (G == 1) {
            // rows 4-15 are zero (no second head): two 16-lane row swaps and one 32-lane swap
            // move the limbs of tiles 4hf+1..4hf+3 into row groups 1-3 of tile 4hf's registers
            const int e = vsh + 7;
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                v4i m;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int a01 = __builtin_amdgcn_permlane16_swap(gacc[4 * hf][r], gacc[4 * hf + 1][r], false, false)[0];
                    const int a23 = __builtin_amdgcn_permlane16_swap(gacc[4 * hf + 2][r], gacc[4 * hf + 3][r], false, false)[0];
                    m[r] = (int)__builtin_amdgcn_permlane32_swap(a01, a23, false, false)[0];
                }
                oacc[hf] += ldexpf(limbs(m), -e);
            }
        } else if (hq < G) {
            const int e = vsh + 7;
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) oacc[nt] += ldexpf(limbs(gacc[nt]), -e);
        }
        // the integer sums replace the weights just read (a wave's LDS operations run in
        // issue order)
        wave_sync();
#pragma unroll
        for (int hd = 0; hd < G; ++hd) {
            S.oci(hd, lane) = 0;
            S.oci(hd, lane + 64) = 0;
        }
        wave_sync();
        value_corrections<G, PG>(S, a, sc, cap, unpack_run(run_c), staged, gc, tok0, lane);
        wave_sync();
        // fold the group's integer sums into the fp32 outputs
        if constexpr (G == 1) {
            ocr[0][0] += ldexpf((float)S.oci(0, lane), -fsh);
            ocr[0][1] += ldexpf((float)S.oci(0, lane + 64), -fsh);
        } else {
#pragma unroll
            for (int hp = 0; hp < G / 2; ++hp) {
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    const unsigned long long T = S.oci2(hp, lane + 64 * c);
                    const int s0 = (int)(uint32_t)T;
                    const int s1 = (int)(uint32_t)(T >> 32) + (s0 < 0 ? 1 : 0);
                    ocr[2 * hp][c] += ldexpf((float)s0, -fsh);
                    ocr[2 * hp + 1][c] += ldexpf((float)s1, -fsh);
                }
            }
        }
        wave_sync();   // (the next group's weights replace the sums)
        gc = gn;
        gn = gnn;
        tab_n = tab_nn;
        fits_c = fits_n;
        run_c = run_n;
    }

#pragma unroll
    for (int hd = 0; hd < G; ++hd) {
        const float v = wave_sum(pb[hd]);
        if (lane == 0) S.pbase[hd] = v;
        S.oc()[hd][lane] = ocr[hd][0];
        S.oc()[hd][lane + 64] = ocr[hd][1];
    }
    wave_sync();
    if (hq < G || G == 1) {
        const int hd = G == 1 ? 0 : hq;
        const int64_t row = (int64_t)s * a.Hq + qh0 + hd;
        const float l = S.l[hd];
#pragma unroll
        for (int nt = 0; nt < NO; ++nt) {
            const int j = (G == 1 ? 4 * nt + hq : nt) * 16 + (lane & 15);
            const float o = S.pbase[hd] + oacc[nt] + S.oc()[hd][j];
            if (a.n_splits == 1) {
                a.out[row * D + j] = (l > 0.0f) ? o / l : 0.0f;
            } else {
                float* pp = a.partial + (row * a.n_splits + split) * (D + 2);
                pp[j] = o;
                if (j == 0) {
                    pp[D] = S.m[hd];
                    pp[D + 1] = l;
                }
            }
        }
    }
}

}  // namespace

// The kernel with on-demand sparse pages is compiled in a translation unit of its own
// (attention_mfma_paged.hip includes this file with OAKEN_ATTN_PAGED_TU defined): in one
// module with the fixed-record kernel it changes the fixed kernel's register allocation.
template <bool PG>
static hipError_t launch_mfma(const AttnArgs& a, hipStream_t st) {
    const int G = a.wave_heads;
    if (G * a.head_parts != a.Hq / a.H) return hipErrorInvalidValue;
    // a range spans at most 32 pages (the lane reads of the page table rely on it)
    if (a.pages_per_split > 32 || a.pages_per_split * P > mfma_score_cap(G)) return hipErrorInvalidValue;
    const size_t shm = (size_t)G * a.pages_per_split * P * sizeof(float);
    const uint32_t grid = attn_grid(a);
    if (grid == 0) return hipErrorInvalidValue;
    if (G == 1)
        hipLaunchKernelGGL((attn_mfma_kernel<1, PG>), dim3(grid), dim3(64), shm, st, a);
    else if (G == 2)
        hipLaunchKernelGGL((attn_mfma_kernel<2, PG>), dim3(grid), dim3(64), shm, st, a);
    else if (G == 4)
        hipLaunchKernelGGL((attn_mfma_kernel<4, PG>), dim3(grid), dim3(64), shm, st, a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

#ifdef OAKEN_ATTN_PAGED_TU
hipError_t launch_attention_mfma_paged(const AttnArgs& a, hipStream_t st) { return launch_mfma<true>(a, st); }
#else
bool mfma_attention_supported(int d, int G) { return d == D && G >= 1 && G <= 8; }

// G = 8 and 4 take four heads per workgroup, 6 and 2 two, the odd counts one.
int mfma_wave_heads(int G) { return G % 4 == 0 ? 4 : (G % 2 == 0 ? 2 : 1); }

// Four heads per workgroup keep 16 pages of scores (the wave's LDS then allows nine
// waves per CU; measured faster on the GQA layers than 15 or 20 pages), the others 32.
int mfma_score_cap(int wave_heads) { return wave_heads == 4 ? 256 : 512; }

hipError_t launch_attention_mfma(const AttnArgs& a, hipStream_t st) {
    return a.spool ? launch_attention_mfma_paged(a, st) : launch_mfma<false>(a, st);
}
#endif

}  // namespace oaken
