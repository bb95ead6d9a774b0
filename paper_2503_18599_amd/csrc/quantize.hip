// Online KV quantization into the paged cache (Oaken Sec. 4.3-4.5, Sec. 5.2
// quantization engine and MMU).
//
// One wave writes one record segment: the new tokens of one sequence that fall into one
// page, for one KV head and one of K/V (a workgroup holds four independent waves).  A
// vector of d elements is spread over d/8 lanes with eight consecutive elements each
// (one 16-byte load), so a wave quantizes 64 / (d/8) vectors at a time: for d = 128 the
// four 16-lane rows of the wave hold four tokens.  Group minima and maxima are taken
// over a lane's eight elements, then across the vector's lanes by DPP, with no LDS round
// trip.  Group selection is compares and selects, so waves never diverge on the value
// distribution.
//
// The lanes of a wave hold their vectors' elements in stream order (slot, then 64-value
// chunk, then index), so a wave-wide prefix sum of per-lane outlier counts places every
// COO entry in the record's stream: the engine's zero-remove step, without branches.
// Outputs are assembled in LDS and leave in wide stores: K rows as dwords straight from
// registers, metadata as dwords, V pages (channel-major) and COO streams in 16-byte
// chunks when the segment starts the page.
#include "oaken_internal.h"

#include <hip/hip_fp16.h>

// The quantizer's codes are a bit-exact contract: one IEEE rounding per operation.
#pragma clang fp contract(off)

namespace oaken {
namespace {

__device__ inline float half_bits_to_float(uint32_t b) {
    return __half2float(__ushort_as_half((uint16_t)b));
}

__device__ inline uint16_t float_to_half_bits(float f) {
    return __half_as_ushort(__float2half_rn(f));
}

// (every lane of these permutations reads a lane of its own group)
template <int C>
__device__ inline int dpp_i(int v) {
    return __builtin_amdgcn_mov_dpp(v, C, 0xf, 0xf, true);
}

// Reductions over the N = 8 or 16 lanes of a vector (aligned lane groups): quad
// butterflies, then the half-row and row mirrors.  Every lane of the group gets the
// result.
constexpr int kQuadXor1 = 0xb1, kQuadXor2 = 0x4e, kRowHalfMirror = 0x141, kRowMirror = 0x140;

template <int N>
__device__ inline uint32_t group_min_u(uint32_t v) {
    v = min(v, (uint32_t)dpp_i<kQuadXor1>((int)v));
    v = min(v, (uint32_t)dpp_i<kQuadXor2>((int)v));
    v = min(v, (uint32_t)dpp_i<kRowHalfMirror>((int)v));
    if constexpr (N == 16) v = min(v, (uint32_t)dpp_i<kRowMirror>((int)v));
    return v;
}
template <int N>
__device__ inline int group_max_i(int v) {
    v = max(v, dpp_i<kQuadXor1>(v));
    v = max(v, dpp_i<kQuadXor2>(v));
    v = max(v, dpp_i<kRowHalfMirror>(v));
    if constexpr (N == 16) v = max(v, dpp_i<kRowMirror>(v));
    return v;
}
// Sum over aligned groups of 8 lanes.
__device__ inline int sum8(int v) {
    v += dpp_i<kQuadXor1>(v);
    v += dpp_i<kQuadXor2>(v);
    v += dpp_i<kRowHalfMirror>(v);
    return v;
}

// Inclusive prefix sum over the wave: DPP row scan, then the rows' totals carried by row
// broadcasts (lane 15 of rows 0 and 2 into rows 1 and 3, then lane 31 into rows 2 and 3).
__device__ inline int wave_incl_scan(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);   // row_bcast:15
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return x;
}

// LDS addresses as plain 32-bit integers (an address that a select picks whole).
typedef __attribute__((address_space(3))) uint8_t lds_byte;
__device__ inline uint32_t off_lds(const void* p) { return (uint32_t)(uintptr_t)(const lds_byte*)p; }
__device__ inline lds_byte& lds_u8(uint32_t a) { return *(lds_byte*)(uintptr_t)a; }

// x + 1 in the lanes of the lane mask c, else x: one add with c as the carry in.
__device__ inline int add_if(int x, uint64_t c) {
    int r;
    uint64_t carry;
    asm("v_addc_co_u32_e64 %0, %1, %2, 0, %3" : "=v"(r), "=s"(carry) : "v"(x), "s"(c));
    return r;
}
// c ? a : b per lane of the lane mask c.
__device__ inline uint32_t pick(uint64_t c, uint32_t a, uint32_t b) {
    uint32_t r;
    asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(b), "v"(a), "s"(c));
    return r;
}

// The lanes of one wave hand LDS data to each other: LDS operations of a wave execute in
// issue order, so only compiler fences are needed.
__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Codes of the eight elements a lane holds of one vector (Eq. 1-4), the vector spread over
// LPV aligned lanes with eight consecutive elements each (m = lane within the vector).
struct LaneCodes {
    uint32_t nib[8];   // the dense nibble (low 4 bits of the code)
    uint32_t cb[8];    // the COO byte of an inner or outer value
    uint64_t out[8];   // lane mask of the lanes whose element e is inner or outer
    int n_out;         // inner and outer values among the eight
    float meta;        // lanes m < 6: field m of the vector's metadata (Min_g, Delta_g)
};

// The thresholds must satisfy lo_o <= lo_i <= hi_i <= hi_o and x must be finite.  Per
// element, with t_o = med3(x, lo_o, hi_o) and t_i = med3(x, lo_i, hi_i) (x clamped to the
// outer and inner intervals): x - t_o is non-zero exactly for outer values, where it is
// the Eq. 4 shifted value, and x - t_i is zero exactly for inner values and the shifted
// value of a middle one (differences of distinct floats never round to zero).  The
// signed value v (x + 0 for inner ones, which turns -0 into +0) then carries the side in
// its sign bit (side = v >= 0) and the group's magnitude a = |v|.
template <int LPV>
__device__ inline LaneCodes quantize_lane(const uint32_t (&w4)[4], float lo_o, float lo_i, float hi_i, float hi_o,
                                          int m, int lane) {
    LaneCodes R;
    // group minima and maxima over the magnitudes' bit patterns (non-negative floats order
    // as integers): an element of another group reads as 0xffffffff, the largest unsigned
    // and the smallest signed key, so one key serves the unsigned minimum and the signed
    // maximum
    float v[8];
    bool outer[8], inner[8];
    uint32_t kmin[3] = {~0u, ~0u, ~0u};
    int kmax[3] = {-1, -1, -1};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float xf = half_bits_to_float((e & 1) ? (w4[e >> 1] >> 16) : (w4[e >> 1] & 0xffffu));
        const float d_o = xf - __builtin_amdgcn_fmed3f(xf, lo_o, hi_o);
        const float d_i = xf - __builtin_amdgcn_fmed3f(xf, lo_i, hi_i);
        const bool o = d_o != 0.0f;                  // Eq. 1, outer
        const bool in = d_i == 0.0f;                 // inner (not shifted)
        v[e] = in ? xf + 0.0f : (o ? d_o : d_i);     // Eq. 4
        outer[e] = o;
        inner[e] = in;
        R.out[e] = __builtin_amdgcn_ballot_w64(d_o != 0.0f) | __builtin_amdgcn_ballot_w64(d_i == 0.0f);
        const uint32_t mb = __float_as_uint(v[e]) & 0x7fffffffu;
        const uint32_t ki = in ? mb : ~0u, km = (o || in) ? ~0u : mb, ko = o ? mb : ~0u;
        kmin[0] = min(kmin[0], ki); kmax[0] = max(kmax[0], (int)ki);
        kmin[1] = min(kmin[1], km); kmax[1] = max(kmax[1], (int)km);
        kmin[2] = min(kmin[2], ko); kmax[2] = max(kmax[2], (int)ko);
    }
    float gmin[3], grng[3];
#pragma unroll
    for (int g = 0; g < 3; ++g) {
        const uint32_t lo = group_min_u<LPV>(kmin[g]);
        const int hi = group_max_i<LPV>(kmax[g]);
        const bool empty = hi < 0;                   // (0, 0) for an empty group
        gmin[g] = empty ? 0.0f : __uint_as_float(lo);
        grng[g] = empty ? 0.0f : __int_as_float(hi) - gmin[g];
    }
    // Eq. 2: lane 2g of the vector forms sigma_g = L/R, lane 2g+1 Delta_g = R/L (its
    // metadata); one correctly rounded division per lane
    const int g6 = (m >> 1) < 3 ? (m >> 1) : 0;
    const bool is_delta = (m & 1) != 0;
    const float Rg = g6 == 0 ? grng[0] : (g6 == 1 ? grng[1] : grng[2]);
    const float Lg = g6 == 1 ? 7.0f : 15.0f;
    float quo = (is_delta ? Rg : Lg) / (is_delta ? Lg : Rg);
    if (!is_delta && Rg == 0.0f) quo = 0.0f;
    const int vbase = lane & ~(LPV - 1);
    float sig[3];
#pragma unroll
    for (int g = 0; g < 3; ++g) sig[g] = __shfl(quo, vbase + 2 * g, 64);
    R.meta = is_delta ? quo : gmin[g6];

    // Eq. 3.  0 <= (a - Min) * sigma < L + 1/2 (a - Min <= R rounds to at most R, and
    // R * fl(L / R) to less than L + 1/2), so adding 2^23 rounds it half-to-even to an
    // integer c in the low bits and no clamp is needed.  The offset-binary code
    // u = side ? 2^b + c : 2^b - 1 - c has the low four bits c ^ (middle ? 8 : 0) when the
    // side is set and their complement otherwise; sg (v's sign spread over the word) is
    // the complement of the side.
    const uint32_t m8 = (uint32_t)(8 * m) & 63u;
    R.n_out = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const bool o = outer[e], in = inner[e];
        const float gm = o ? gmin[2] : (in ? gmin[0] : gmin[1]);
        const float gs = o ? sig[2] : (in ? sig[0] : sig[1]);
        const float r = (fabsf(v[e]) - gm) * gs + 0x1p23f;
        const uint32_t sg = (uint32_t)(__float_as_int(v[e]) >> 31);
        R.nib[e] = (__float_as_uint(r) ^ ((o || in) ? 0u : 8u) ^ sg) & 15u;
        R.cb[e] = (((o ? 0xc0u : 0x80u) | m8) + (uint32_t)e) ^ (sg & 0x80u);
        R.n_out = add_if(R.n_out, R.out[e]);
    }
    return R;
}

// One wave's staging area: the segment's COO bytes (from the segment's first entry),
// V nibbles one byte per element, fp16 metadata and per-chunk counts by slot, and the
// record's sparse page ids (on-demand pages).
template <int D>
struct WaveBuf {
    __align__(16) uint8_t coo[kPage * D + 256];   // (+ one spare byte per lane, 4 apart)
    __align__(16) uint8_t vn[kPage][D];
    __align__(16) uint16_t meta[kPage][6];
    uint8_t cnt[kPage][D / 64];
    int32_t tab[kPage * D / kSparsePage];
};

constexpr int kWavesPerGroup = 4;

template <int D, bool PG>
__global__ __launch_bounds__(64 * kWavesPerGroup) void quantize_kernel(QuantArgs a) {
    constexpr int NC = D / 64;                 // 64-value chunks per vector
    constexpr int LPV = D / 8;                 // lanes per vector
    constexpr int VPP = 64 / LPV;              // vectors per pass
    constexpr int NPASS = kPage / VPP;         // passes for a whole page
    constexpr Layout LY = PG ? make_layout_paged(kPage, D) : make_layout(kPage, D);
    constexpr int NT = kPage * D / kSparsePage;   // sparse pages a record can need
    constexpr int CAP = kPage * D;                // COO capacity of a record

    __shared__ WaveBuf<D> bufs[kWavesPerGroup];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    WaveBuf<D>& W = bufs[wave];

    const int hw = (int)blockIdx.z * kWavesPerGroup + wave;   // (KV head, K|V)
    if (hw >= 2 * a.H) return;
    const int h = hw >> 1, which = hw & 1;
    const int s = blockIdx.y;
    const int row0 = a.cu_tokens[s];
    const int n_new = a.cu_tokens[s + 1] - row0;
    const int pos0 = a.start_pos[s];
    const int page = pos0 / kPage + (int)blockIdx.x;
    const int t_lo = max(pos0, page * kPage);
    const int t_hi = min(pos0 + n_new, (page + 1) * kPage);
    if (n_new <= 0 || t_lo >= t_hi || page >= a.max_blocks) return;   // uniform per wave
    const int blk = a.block_table[(int64_t)s * a.max_blocks + page];
    if (blk < 0 || blk >= a.num_blocks) return;
    const int slot0 = t_lo - page * kPage;     // first slot written
    const int nslots = t_hi - t_lo;            // 1 .. 16
    uint8_t* rec = a.pool + (((int64_t)blk * a.H + h) * 2 + which) * a.stride;

    // ---- loads: every pass's input first, then what this call keeps from the record --
    const int r = lane / LPV, m = lane % LPV;  // vector within a pass, lane within the vector
    const uint16_t* xsrc = which ? a.v_new : a.k_new;
    const int64_t rbase = (int64_t)row0 + (t_lo - pos0);
    uint4 xin[NPASS];
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
        const int i = p * VPP + r;
        const int64_t row = rbase + (i < nslots ? i : 0);   // (past the segment: its first row)
        xin[p] = *reinterpret_cast<const uint4*>(xsrc + (row * a.H + h) * D + 8 * m);
    }
    // the COO bytes of the record's earlier slots: this segment's stream starts after them
    int pre = 0;
    if (slot0 > 0) {
        const int c = lane < slot0 * NC ? (int)rec[LY.counts + lane] : 0;
        pre = __builtin_amdgcn_readlane(wave_incl_scan(c), 63);
        pre = min(pre, CAP);
    }
    const int tab_pre = (PG && lane < NT) ? reinterpret_cast<const int32_t*>(rec + LY.sparse)[lane] : 0;
    // V starting at an odd slot shares its first byte per channel with the slot before
    uint32_t old_b[NC];
#pragma unroll
    for (int k = 0; k < NC; ++k) old_b[k] = 0;
    if (which == 1 && (slot0 & 1)) {
#pragma unroll
        for (int k = 0; k < NC; ++k) old_b[k] = rec[LY.dense + (lane + 64 * k) * (kPage / 2) + (slot0 >> 1)];
    }

    const float* th = a.thr + (h * 2 + which) * 4;
    const float lo_o = th[0], lo_i = th[1], hi_i = th[2], hi_o = th[3];

    // ---- quantize, pass by pass (Eq. 1-4) ----------------------------------------
    int off = pre;   // stream offset of the pass's first entry (wave-uniform)
    const int npass = (nslots + VPP - 1) / VPP;
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
        if (p >= npass) break;   // (uniform)
        const int i = p * VPP + r;
        const bool valid = i < nslots;
        const int t = slot0 + i;
        const uint32_t w4[4] = {xin[p].x, xin[p].y, xin[p].z, xin[p].w};

        const LaneCodes Q = quantize_lane<LPV>(w4, lo_o, lo_i, hi_i, hi_o, m, lane);
        const uint32_t(&nib)[8] = Q.nib;
        const int cnt = valid ? Q.n_out : 0;

        // dense nibbles: K row dwords go out directly; V nibbles are staged by slot
        if (which == 0) {
            uint32_t kw = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e) kw |= nib[e] << (4 * e);
            if (valid) *reinterpret_cast<uint32_t*>(rec + LY.dense + t * (D / 2) + 4 * m) = kw;
        } else if (valid) {
            const uint32_t lo = nib[0] | (nib[1] << 8) | (nib[2] << 16) | (nib[3] << 24);
            const uint32_t hi = nib[4] | (nib[5] << 8) | (nib[6] << 16) | (nib[7] << 24);
            *reinterpret_cast<uint2*>(&W.vn[t][8 * m]) = make_uint2(lo, hi);
        }
        // metadata: lane m < 6 holds field m of the slot: Min_g (even), Delta_g (odd)
        if (valid && m < 6) W.meta[t][m] = float_to_half_bits(Q.meta);

        // COO entries: positions from a wave-wide prefix sum of the lanes' counts
        const int incl = wave_incl_scan(cnt);
        const int c8 = sum8(cnt);   // entries of the lane's 64-value chunk
        if (valid && (m & 7) == 0) W.cnt[t][m >> 3] = (uint8_t)c8;
        // every element stores its byte: entries at their stream positions (below CAP:
        // a segment has at most CAP entries), the others in the lane's own spare byte
        const uint64_t vmask = __builtin_amdgcn_ballot_w64(valid);
        const uint32_t spare = off_lds(&W.coo[CAP + 4 * lane]);
        int at = (int)off_lds(&W.coo[0]) + off - pre + incl - cnt;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint64_t put = vmask & Q.out[e];
            lds_u8(pick(put, (uint32_t)at, spare)) = (uint8_t)Q.cb[e];
            at = add_if(at, put);
        }
        off += __builtin_amdgcn_readlane(incl, 63);
    }
    wave_sync();

    // ---- stores ------------------------------------------------------------------
    const int n = min(off, CAP) - pre;   // COO bytes of this segment
    if (lane < nslots * NC) rec[LY.counts + slot0 * NC + lane] = W.cnt[slot0 + lane / NC][lane % NC];
    if (lane < 3 * nslots)
        reinterpret_cast<uint32_t*>(rec + LY.meta + slot0 * 12)[lane] =
            reinterpret_cast<const uint32_t*>(&W.meta[slot0][0])[lane];
    if (which == 1) {
        if (slot0 == 0) {
            // whole pairs: lane l writes channels 2l and 2l+1 (16 bytes); slots past the
            // segment read as zero nibbles (writing a slot invalidates the later ones)
            if (2 * lane < D) {
                uint32_t wq[kPage];
#pragma unroll
                for (int tt = 0; tt < kPage; ++tt)
                    wq[tt] = tt < nslots ? (uint32_t)*reinterpret_cast<const uint16_t*>(&W.vn[tt][2 * lane]) : 0u;
                uint32_t d2[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    // pairs 2k and 2k+1: low byte channel 2l, high byte channel 2l+1
                    const uint32_t c0 = wq[4 * k] | (wq[4 * k + 1] << 4);
                    const uint32_t c1 = wq[4 * k + 2] | (wq[4 * k + 3] << 4);
                    d2[k] = c0 | (c1 << 16);
                }
                uint4 ov;
                ov.x = __builtin_amdgcn_perm(d2[1], d2[0], 0x06040200u);   // channel 2l, pairs 0-3
                ov.y = __builtin_amdgcn_perm(d2[3], d2[2], 0x06040200u);   // pairs 4-7
                ov.z = __builtin_amdgcn_perm(d2[1], d2[0], 0x07050301u);   // channel 2l+1
                ov.w = __builtin_amdgcn_perm(d2[3], d2[2], 0x07050301u);
                *reinterpret_cast<uint4*>(rec + LY.dense + 16 * lane) = ov;
            }
        } else {
            // a segment starting inside the page: byte by byte, the first byte keeping the
            // earlier slot's low nibble when the segment starts at an odd slot
            const int p_lo = slot0 >> 1, p_hi = (slot0 + nslots - 1) >> 1;
#pragma unroll
            for (int k = 0; k < NC; ++k) {
                const int j = lane + 64 * k;
                for (int q = p_lo; q <= p_hi; ++q) {
                    const int te = 2 * q, to = te + 1;
                    const uint32_t lo_n = te >= slot0 ? W.vn[te][j] : (old_b[k] & 0x0fu);
                    const uint32_t hi_n = to < slot0 + nslots ? W.vn[to][j] : 0u;
                    rec[LY.dense + j * (kPage / 2) + q] = (uint8_t)(lo_n | (hi_n << 4));
                }
            }
        }
    }

    // ---- COO stream ----------------------------------------------------------------
    if constexpr (PG) {
        // Sparse pages on demand (Sec. 5.2 MMU): the record's stream now needs
        // ceil(used / 256) pages; the ones it does not hold yet are reserved from the
        // free list with a compare-and-swap that only succeeds while enough pages are
        // free (so the count never passes below what is really free), and entered in its
        // table (entry = 1 + page id, 0 = none held).  A list without enough pages sets
        // the overflow flag and leaves those pages out (their bytes are not written).
        const int p_new = min(NT, (pre + n + kSparsePage - 1) / kSparsePage);
        const bool need = lane < p_new && tab_pre == 0;
        const uint64_t nm = __ballot(need);
        const int k = __popcll(nm);
        int top = -1;
        if (k > 0 && lane == 0) {
            int cur = __hip_atomic_load(&a.sfree[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            while (true) {
                if (cur < k || cur > a.spages) {   // (a consistent list never exceeds the pool)
                    atomicOr(&a.sfree[1], 1);
                    break;
                }
                const int seen = atomicCAS(&a.sfree[0], cur, cur - k);
                if (seen == cur) {
                    top = cur;
                    break;
                }
                cur = seen;   // another record took pages first: retry with the new count
            }
        }
        top = __shfl(top, 0, 64);
        int entry = tab_pre;
        if (need && top >= k) {
            const int rk = __popcll(nm & ((1ull << lane) - 1ull));
            entry = 1 + a.sfree[2 + top - k + rk];
            reinterpret_cast<int32_t*>(rec + LY.sparse)[lane] = entry;
        }
        if (lane < NT) W.tab[lane] = entry - 1;
        wave_sync();
    }
    auto coo_dst = [&](int o) -> uint8_t* {
        if constexpr (PG) {
            const int id = W.tab[o / kSparsePage];
            return (id >= 0 && id < a.spages) ? a.spool + (int64_t)id * kSparsePage + (o % kSparsePage) : nullptr;
        } else {
            return rec + LY.sparse + o;
        }
    };
    if (n > 0) {
        if ((pre & 15) == 0) {
            // 16-byte chunks (never straddling a sparse page); bytes past the stream are
            // written as zero
            for (int c = lane; c * 16 < n; c += 64) {
                uint4 v = *reinterpret_cast<const uint4*>(&W.coo[16 * c]);
                const int nb = n - 16 * c;
                if (nb < 16) {
                    uint32_t* vw = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int keep = min(max(nb - 4 * q, 0), 4);
                        vw[q] = keep == 4 ? vw[q] : (vw[q] & ((1u << (8 * keep)) - 1u));
                    }
                }
                uint8_t* dst = coo_dst(pre + 16 * c);
                if (dst) *reinterpret_cast<uint4*>(dst) = v;
            }
        } else {
            for (int b = lane; b < n; b += 64) {
                uint8_t* dst = coo_dst(pre + b);
                if (dst) *dst = W.coo[b];
            }
        }
    }
}

// Sum over the N = 8 or 16 lanes of a vector (aligned lane groups); every lane gets it.
template <int N>
__device__ inline int group_sum(int v) {
    v += dpp_i<kQuadXor1>(v);
    v += dpp_i<kQuadXor2>(v);
    v += dpp_i<kRowHalfMirror>(v);
    if constexpr (N == 16) v += dpp_i<kRowMirror>(v);
    return v;
}
// Inclusive prefix sum over the N lanes of a vector (m = lane within it): row shifts, each
// added only where its source lies in the same vector.
template <int N>
__device__ inline int group_incl_scan(int x, int m) {
    int y;
    y = __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += m >= 1 ? y : 0;
    y = __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x += m >= 2 ? y : 0;
    y = __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x += m >= 4 ? y : 0;
    if constexpr (N == 16) {
        y = __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
        x += m >= 8 ? y : 0;
    }
    return x;
}

// One new token per sequence (the decode step), fixed-capacity records: every vector
// (sequence, KV head, K|V) on its own d/8 lanes, so a wave quantizes 64 / (d/8) vectors
// at once instead of one.  Same codes, stream order and record writes as quantize_kernel
// for a segment of one slot; the vector's COO offset comes from a prefix sum over its
// own lanes and the record's counts of the earlier slots.  All lanes stay active through
// the lane exchanges; vectors without a token only skip their loads and stores.
// A workgroup takes (KV head, K|V) vectors of one sequence (grid x: the sequence), so the
// sequence's row, position and block are uniform loads.
template <int D>
__global__ __launch_bounds__(256) void quantize_token_kernel(QuantArgs a) {
    constexpr int NC = D / 64, LPV = D / 8, VPW = 64 / LPV;
    constexpr Layout LY = make_layout(kPage, D);
    constexpr int CAP = kPage * D;
    const int lane = threadIdx.x & 63, r = lane / LPV, m = lane % LPV;
    const int s = (int)blockIdx.x;
    const int hw_l = ((int)blockIdx.y * (int)(blockDim.x >> 6) + (int)(threadIdx.x >> 6)) * VPW + r;
    const bool in_range = hw_l < 2 * a.H;
    const int hw = in_range ? hw_l : 0;
    const int h = hw >> 1, which = hw & 1;
    // The loads form three dependent levels, each issued whole before its first use:
    // the sequence's row and position; its block and the input vector; what the record
    // keeps from earlier slots.
    const int row = a.cu_tokens[s], row_end = a.cu_tokens[s + 1], pos = a.start_pos[s];
    const float* th = a.thr + hw * 4;
    const float lo_o = th[0], lo_i = th[1], hi_i = th[2], hi_o = th[3];
    const int page = pos / kPage, slot = pos % kPage;
    const bool seq_ok = row_end - row == 1 && pos >= 0 && page < a.max_blocks;   // (uniform)
    const int blk = seq_ok ? a.block_table[(int64_t)s * a.max_blocks + page] : -1;
    uint4 x = make_uint4(0, 0, 0, 0);
    if (in_range && seq_ok)   // (beside the block load, not after it)
        x = *reinterpret_cast<const uint4*>((which ? a.v_new : a.k_new) + ((int64_t)row * a.H + h) * D + 8 * m);
    const bool ok = in_range && seq_ok && blk >= 0 && blk < a.num_blocks;
    uint8_t* rec = a.pool + (((int64_t)(ok ? blk : 0) * a.H + h) * 2 + which) * a.stride;
    // COO bytes of the record's earlier slots (2 count bytes per lane cover 2 * LPV >=
    // slot * NC), and V at an odd slot: the bytes it shares with the slot before
    int c = 0;
    uint32_t old_b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) old_b[e] = 0;
    if (ok) {
        const int b0 = 2 * m, b1 = 2 * m + 1;
        c = (b0 < slot * NC ? (int)rec[LY.counts + b0] : 0) + (b1 < slot * NC ? (int)rec[LY.counts + b1] : 0);
        if (which == 1 && (slot & 1)) {
#pragma unroll
            for (int e = 0; e < 8; ++e) old_b[e] = rec[LY.dense + (8 * m + e) * (kPage / 2) + (slot >> 1)];
        }
    }
    const int pre = min(group_sum<LPV>(c), CAP);

    const uint32_t w4[4] = {x.x, x.y, x.z, x.w};
    const LaneCodes Q = quantize_lane<LPV>(w4, lo_o, lo_i, hi_i, hi_o, m, lane);
    const int cnt = Q.n_out;
    const int incl = group_incl_scan<LPV>(cnt, m);
    const int c8 = group_sum<8>(cnt);   // entries of the lane's 64-value chunk
    if (!ok) return;   // (no lane exchange below)

    if (which == 0) {
        uint32_t kw = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) kw |= Q.nib[e] << (4 * e);
        *reinterpret_cast<uint32_t*>(rec + LY.dense + slot * (D / 2) + 4 * m) = kw;
    } else {
        // channel-major: channel j's byte slot / 2, low nibble the even slot; writing an
        // even slot clears the odd one after it
#pragma unroll
        for (int e = 0; e < 8; ++e)
            rec[LY.dense + (8 * m + e) * (kPage / 2) + (slot >> 1)] =
                (uint8_t)((slot & 1) ? ((old_b[e] & 0x0fu) | (Q.nib[e] << 4)) : Q.nib[e]);
    }
    if (m < 6) reinterpret_cast<uint16_t*>(rec + LY.meta + slot * 12)[m] = float_to_half_bits(Q.meta);
    if ((m & 7) == 0) rec[LY.counts + slot * NC + (m >> 3)] = (uint8_t)c8;
    int p = pre + incl - cnt;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        if ((Q.out[e] >> lane) & 1) {
            if (p < CAP) rec[LY.sparse + p] = (uint8_t)Q.cb[e];
            ++p;
        }
    }
}

}  // namespace

hipError_t launch_quantize(const QuantArgs& a, int d, int max_new_per_seq, hipStream_t st) {
    const bool pg = a.spool != nullptr;
    if (max_new_per_seq == 1 && !pg) {
        // the decode step: one vector per d/8 lanes, the sequences along x
        const int per_block = 4 * (64 / (d / 8));
        const dim3 grid((uint32_t)a.n_seqs, (uint32_t)((2 * a.H + per_block - 1) / per_block));
        if (d == 64)
            hipLaunchKernelGGL(quantize_token_kernel<64>, grid, dim3(256), 0, st, a);
        else if (d == 128)
            hipLaunchKernelGGL(quantize_token_kernel<128>, grid, dim3(256), 0, st, a);
        else
            return hipErrorInvalidValue;
        return hipGetLastError();
    }
    // pages a run of n tokens can touch: (n + P - 2) / P + 1 (one for a single token)
    const int segs = (max_new_per_seq + kPage - 2) / kPage + 1;
    dim3 grid(segs, a.n_seqs, (2 * a.H + kWavesPerGroup - 1) / kWavesPerGroup);
    dim3 block(64 * kWavesPerGroup);
    if (d == 64 && !pg)
        hipLaunchKernelGGL((quantize_kernel<64, false>), grid, block, 0, st, a);
    else if (d == 128 && !pg)
        hipLaunchKernelGGL((quantize_kernel<128, false>), grid, block, 0, st, a);
    else if (d == 64)
        hipLaunchKernelGGL((quantize_kernel<64, true>), grid, block, 0, st, a);
    else if (d == 128)
        hipLaunchKernelGGL((quantize_kernel<128, true>), grid, block, 0, st, a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace oaken
