// Online KV quantization into the paged cache (Oaken Sec. 4.3-4.5, Sec. 5.2
// quantization engine).
//
// One workgroup covers the new tokens of one sequence that fall into one page, for
// one KV head and one of K/V; each wave64 quantizes one token's vector.  Lane l owns
// elements j = 64*c + l, so a wave's ballot over chunk c is exactly that chunk's
// outlier mask: its popcount is the chunk count and mbcnt gives each outlier's slot
// in the COO stream (the zero-remove step of the engine) without any branch.
// Group selection is done with compares and selects, so waves never diverge on the
// value distribution.
#include "oaken_internal.h"

#include <hip/hip_fp16.h>

// The quantizer's codes are a bit-exact contract: one IEEE rounding per operation.
#pragma clang fp contract(off)

namespace oaken {
namespace {

__device__ inline float half_bits_to_float(uint16_t b) {
    return __half2float(__ushort_as_half(b));
}

__device__ inline uint16_t float_to_half_bits(float f) {
    return __half_as_ushort(__float2half_rn(f));
}

// Wave reductions: a DPP shift-scan within each row of 16 lanes leaves the row's result
// in its lane 15; the four row results combine through readlane (no LDS round trips).
template <typename Op>
__device__ inline float wave_reduce(float v, float ident, Op op) {
    const int id = __float_as_int(ident);
    v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(id, __float_as_int(v), 0x111, 0xf, 0xf, false)));
    v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(id, __float_as_int(v), 0x112, 0xf, 0xf, false)));
    v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(id, __float_as_int(v), 0x114, 0xf, 0xf, false)));
    v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(id, __float_as_int(v), 0x118, 0xf, 0xf, false)));
    const int x = __float_as_int(v);
    return op(op(__int_as_float(__builtin_amdgcn_readlane(x, 15)), __int_as_float(__builtin_amdgcn_readlane(x, 31))),
              op(__int_as_float(__builtin_amdgcn_readlane(x, 47)), __int_as_float(__builtin_amdgcn_readlane(x, 63))));
}

__device__ inline float wave_min(float v) {
    return wave_reduce(v, INFINITY, [](float p, float q) { return fminf(p, q); });
}

__device__ inline float wave_max(float v) {
    return wave_reduce(v, -INFINITY, [](float p, float q) { return fmaxf(p, q); });
}

// Inclusive prefix sum over the wave (DPP row scan, then the rows' totals).
__device__ inline int wave_incl_scan(int x, int lane) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);
    const int r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31);
    const int r2 = __builtin_amdgcn_readlane(x, 47);
    const int row = lane >> 4;
    return x + (row == 0 ? 0 : row == 1 ? r0 : row == 2 ? r0 + r1 : r0 + r1 + r2);
}

template <int D, bool PG>
__global__ __launch_bounds__(1024) void quantize_kernel(QuantArgs a) {
    constexpr int NC = D / 64;           // 64-value chunks per vector
    constexpr Layout LY = PG ? make_layout_paged(kPage, D) : make_layout(kPage, D);
    constexpr int NT = kPage * D / kSparsePage;   // sparse pages a record can need

    __shared__ uint8_t s_counts[kPage][NC];
    __shared__ uint8_t s_vnib[kPage][D];
    __shared__ __align__(16) uint8_t s_krow[kPage][D / 2];
    __shared__ int s_tab[NT];            // the record's sparse page ids (on-demand pages)

    const int s = blockIdx.y;
    const int h = blockIdx.z >> 1;
    const int which = blockIdx.z & 1;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;

    const int row0 = a.cu_tokens[s];
    const int n_new = a.cu_tokens[s + 1] - row0;
    const int pos0 = a.start_pos[s];
    const int page = pos0 / kPage + (int)blockIdx.x;
    const int t_lo = max(pos0, page * kPage);
    const int t_hi = min(pos0 + n_new, (page + 1) * kPage);
    if (n_new <= 0 || t_lo >= t_hi || page >= a.max_blocks) return;   // uniform per block
    const int blk = a.block_table[(int64_t)s * a.max_blocks + page];
    if (blk < 0 || blk >= a.num_blocks) return;

    const int slot0 = t_lo - page * kPage;
    const int nslots = t_hi - t_lo;
    uint8_t* rec = a.pool + (((int64_t)blk * a.H + h) * 2 + which) * a.stride;
    const bool active = wave < nslots;
    const int slot = slot0 + wave;

    // Reads that do not depend on this call's values go out first, so that their latency
    // overlaps the quantization: the COO counts of the record's earlier slots, and (values,
    // when the call starts at an odd slot) the bytes the previous token shares with it.
    int pre_cnt = 0;
    if (lane < slot0) {
#pragma unroll
        for (int c = 0; c < NC; ++c) pre_cnt += rec[LY.counts + lane * NC + c];
    }
    // (on-demand pages: the record's page table, for the pages it already holds)
    const int tab_pre = (PG && lane < NT) ? reinterpret_cast<const int32_t*>(rec + LY.sparse)[lane] : 0;
    uint8_t old_b[D / 64];
#pragma unroll
    for (int k = 0; k < D / 64; ++k) old_b[k] = 0;
    if (which == 1 && (slot0 & 1) && wave == 0) {
#pragma unroll
        for (int k = 0; k < D / 64; ++k) old_b[k] = rec[LY.dense + (lane + 64 * k) * (kPage / 2) + (slot0 >> 1)];
    }

    // ---- quantize this wave's vector (Eq. 1-4) -------------------------------------
    const float* th = a.thr + (h * 2 + which) * 4;
    const float lo_o = th[0], lo_i = th[1], hi_i = th[2], hi_o = th[3];

    float av[NC];
    int grp[NC];
    bool side[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) { av[c] = 0.0f; grp[c] = 1; side[c] = false; }
    float mn[3] = {INFINITY, INFINITY, INFINITY};
    float mx[3] = {-INFINITY, -INFINITY, -INFINITY};
    if (active) {
        const int row = row0 + (page * kPage + slot - pos0);
        const uint16_t* x = (which ? a.v_new : a.k_new) + ((int64_t)row * a.H + h) * D;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const float xf = half_bits_to_float(x[c * 64 + lane]);
            const bool outer = (xf < lo_o) || (xf > hi_o);
            const bool middle = !outer && ((xf < lo_i) || (xf > hi_i));
            const int g = outer ? 2 : (middle ? 1 : 0);
            const bool sd = outer ? (xf > hi_o) : (middle ? (xf > hi_i) : (xf >= 0.0f));
            const float shift = outer ? (sd ? hi_o : lo_o) : (middle ? (sd ? hi_i : lo_i) : 0.0f);
            const float mag = (g == 0) ? fabsf(xf) : fabsf(xf - shift);
            av[c] = mag;
            grp[c] = g;
            side[c] = sd;
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                mn[k] = (g == k) ? fminf(mn[k], mag) : mn[k];
                mx[k] = (g == k) ? fmaxf(mx[k], mag) : mx[k];
            }
        }
    }
    float gmin[3], grange[3], gsig[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        float lo = wave_min(mn[k]);
        float hi = wave_max(mx[k]);
        if (!(hi >= lo)) { lo = 0.0f; hi = 0.0f; }   // empty group
        const float levels = (k == 1) ? 7.0f : 15.0f;
        gmin[k] = lo;
        grange[k] = hi - lo;
        gsig[k] = (grange[k] == 0.0f) ? 0.0f : levels / grange[k];
    }

    uint8_t nib[NC];
    uint8_t coo[NC];
    uint64_t omask[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int g = grp[c];
        const int lv = (g == 1) ? 7 : 15;
        const float gm = (g == 0) ? gmin[0] : ((g == 1) ? gmin[1] : gmin[2]);
        const float gs = (g == 0) ? gsig[0] : ((g == 1) ? gsig[1] : gsig[2]);
        const float sh = av[c] - gm;
        const float sc = sh * gs;
        int code = (int)rintf(sc);
        code = min(max(code, 0), lv);
        const int u = side[c] ? (lv + 1) + code : lv - code;
        nib[c] = (uint8_t)(u & 15);
        coo[c] = (uint8_t)(((u >> 4) << 7) | ((g == 2) << 6) | lane);
        omask[c] = __ballot(active && g != 1);
    }
    if (active && lane == 0) {
#pragma unroll
        for (int c = 0; c < NC; ++c) s_counts[slot][c] = (uint8_t)__popcll(omask[c]);
    }
    __syncthreads();

    // sparse start of this slot: the counts of the earlier slots (slots before this call's
    // first one live in the record), as a prefix sum with lane = slot
    int base = 0;
    {
        int cnt = 0;
        if (lane < kPage) {
            if (lane < slot0) {
                cnt = pre_cnt;
            } else if (lane < slot0 + nslots) {
#pragma unroll
                for (int c = 0; c < NC; ++c) cnt += s_counts[lane][c];
            }
        }
        const int incl = wave_incl_scan(cnt, lane);
        base = __shfl(incl - cnt, slot < kPage ? slot : 0, 64);
        if constexpr (PG) {
            // Sparse pages on demand (Sec. 5.2 MMU): the record's COO stream now needs
            // ceil(new_used / 256) pages; wave 0 pops the ones the record does not hold
            // yet from the free list and enters them in its table (entry = 1 + page id,
            // 0 = none held).  An empty list sets the overflow flag and leaves those pages
            // out (their bytes are not written).
            const int new_used = __shfl(incl, slot0 + nslots - 1, 64);
            const int p_new = (new_used + kSparsePage - 1) / kSparsePage;
            if (wave == 0) {
                const bool need = lane < p_new && tab_pre == 0;
                const uint64_t nm = __ballot(need);
                const int k = __popcll(nm);
                int t = 0;
                if (k > 0 && lane == 0) {
                    t = atomicSub(&a.sfree[0], k);
                    if (t < k) {              // not enough pages: give the count back
                        atomicAdd(&a.sfree[0], k);
                        atomicOr(&a.sfree[1], 1);
                    }
                }
                t = __shfl(t, 0, 64);
                int entry = tab_pre;
                if (need && t >= k && t <= a.spages) {   // (a consistent list never exceeds the pool)
                    const int r = __popcll(nm & ((1ull << lane) - 1ull));
                    entry = 1 + a.sfree[2 + t - k + r];
                    reinterpret_cast<int32_t*>(rec + LY.sparse)[lane] = entry;
                }
                if (lane < NT) s_tab[lane] = entry - 1;
            }
            __syncthreads();
        }
    }
    if (active) {
        const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        int off = base;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            if ((omask[c] >> lane) & 1ull) {
                const int o = off + __popcll(omask[c] & below);
                if constexpr (PG) {
                    const int id = s_tab[o / kSparsePage];
                    if (id >= 0 && id < a.spages)
                        a.spool[(int64_t)id * kSparsePage + (o % kSparsePage)] = coo[c];
                } else {
                    rec[LY.sparse + o] = coo[c];
                }
            }
            off += __popcll(omask[c]);
        }
        if (lane < NC) rec[LY.counts + slot * NC + lane] = s_counts[slot][lane];
        if (lane < 6) {
            const int k = lane >> 1;
            const float lv = (k == 1) ? 7.0f : 15.0f;
            const float gm = (k == 0) ? gmin[0] : ((k == 1) ? gmin[1] : gmin[2]);
            const float gr = (k == 0) ? grange[0] : ((k == 1) ? grange[1] : grange[2]);
            const uint16_t hb = (lane & 1) ? float_to_half_bits(gr / lv) : float_to_half_bits(gm);
            *reinterpret_cast<uint16_t*>(rec + LY.meta + slot * 12 + lane * 2) = hb;
        }
        if (which == 0) {
            // K: token-major, element j at byte slot*D/2 + j/2, low nibble = even j; the
            // row is assembled in LDS and leaves in dwords below
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int hi_n = __builtin_amdgcn_update_dpp(0, (int)nib[c], 0x101, 0xf, 0xf, false);   // lane + 1
                if ((lane & 1) == 0) s_krow[slot][(c * 64 + lane) / 2] = (uint8_t)(nib[c] | (hi_n << 4));
            }
        } else {
#pragma unroll
            for (int c = 0; c < NC; ++c) s_vnib[slot][c * 64 + lane] = nib[c];
        }
    }
    __syncthreads();

    if (which == 0) {
        // K rows of this call's slots: one contiguous, 4-byte aligned range
        const uint32_t* src = reinterpret_cast<const uint32_t*>(&s_krow[slot0][0]);
        uint32_t* dst = reinterpret_cast<uint32_t*>(rec + LY.dense + slot0 * (D / 2));
        for (int i = threadIdx.x; i < nslots * (D / 8); i += blockDim.x) dst[i] = src[i];
    } else {
        // V: channel-major, element j of slot t at byte j*P/2 + t/2, low nibble = even t.
        // The first pair (which may keep an earlier token's even nibble) is written by wave
        // 0, one channel per lane; the later pairs by all threads, consecutive threads on
        // consecutive bytes of a channel row.
        const int p_lo = slot0 >> 1, p_hi = (slot0 + nslots - 1) >> 1;
        if (wave == 0) {
            const int te = 2 * p_lo, to = te + 1;
            const bool has_e = te >= slot0;
            const bool has_o = to < slot0 + nslots;
#pragma unroll
            for (int k = 0; k < D / 64; ++k) {
                const int j = lane + 64 * k;
                const uint8_t lo_n = has_e ? s_vnib[te][j] : (uint8_t)(old_b[k] & 0x0f);
                const uint8_t hi_n = has_o ? (uint8_t)(s_vnib[to][j] << 4) : (uint8_t)0;
                rec[LY.dense + j * (kPage / 2) + p_lo] = (uint8_t)(lo_n | hi_n);
            }
        }
        const int npairs = p_hi - p_lo;   // pairs after the first
        for (int i = threadIdx.x; i < npairs * D; i += blockDim.x) {
            const int j = i / npairs;
            const int p = p_lo + 1 + i % npairs;
            const int te = 2 * p, to = 2 * p + 1;
            const bool has_o = to < slot0 + nslots;
            rec[LY.dense + j * (kPage / 2) + p] = has_o ? (uint8_t)(s_vnib[te][j] | (s_vnib[to][j] << 4))
                                                        : s_vnib[te][j];
        }
    }
}

}  // namespace

hipError_t launch_quantize(const QuantArgs& a, int d, int max_new_per_seq, hipStream_t st) {
    const int waves = max(1, min(kPage, max_new_per_seq));
    // pages a run of n tokens can touch: (n + P - 2) / P + 1 (one for a single token)
    const int segs = (max_new_per_seq + kPage - 2) / kPage + 1;
    dim3 grid(segs, a.n_seqs, a.H * 2);
    dim3 block(64 * waves);
    const bool pg = a.spool != nullptr;
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
