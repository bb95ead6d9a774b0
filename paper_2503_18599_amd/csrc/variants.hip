// Group-count variants of the quantizer, for the number-of-groups study (Sec. 6.2):
// two groups (COO entry = sign, pad bit, 6-bit index), four and five groups (two outer
// levels and one or two inner levels; 9-bit COO entries stored in 16 bits) and the
// four- and five-group encodings with 4-bit outliers (the sign moves into the nibble,
// the COO entry keeps 8 bits).  Groups are numbered from the inside out: innermost
// (not shifted), inner a (shifted by the innermost boundary on its side), middle
// (shifted by the inner boundary, or not shifted when there is no inner group), outer a,
// outer b (each shifted by its own inner boundary), as Eq. 4 shifts the three groups.
//
// These encodings are for measuring accuracy against effective bits; they write flat
// per-vector buffers rather than page records.  One wave64 handles one vector of
// d = 64 * NC values; lane l owns elements 64 * c + l, so the ballot over chunk c is the
// chunk's outlier mask and its prefix popcount is each outlier's slot in the stream.
#include "oaken_internal.h"

#include <hip/hip_fp16.h>

// Codes are a bit-exact contract: one IEEE rounding per operation.
#pragma clang fp contract(off)

namespace oaken {

VariantInfo variant_info(int variant) {
    static const int tab[6][3] = {{1, 1, 4}, {1, 0, 4}, {2, 1, 4}, {2, 2, 4}, {2, 1, 3}, {2, 2, 3}};
    VariantInfo v{};
    if (variant < 0 || variant > 5) return v;
    v.n_out = tab[variant][0];
    v.n_in = tab[variant][1];
    v.out_bits = tab[variant][2];
    v.rank_bits = (v.n_out + v.n_in) <= 2 ? 1 : 2;
    v.coo_bits = 6 + v.rank_bits + (v.out_bits == 4 ? 1 : 0);
    v.coo_bytes = v.coo_bits <= 8 ? 1 : 2;
    v.groups = v.n_in + 1 + v.n_out;
    return v;
}

namespace {

constexpr int kMaxGroups = 5;
constexpr int kWaves = 4;   // vectors per workgroup

__device__ inline float h2f(uint16_t b) { return __half2float(__ushort_as_half(b)); }
__device__ inline uint16_t f2h(float f) { return __half_as_ushort(__float2half_rn(f)); }

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

// The eight boundaries: lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa, hi_ob.
struct Bounds {
    float lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa, hi_ob;
};
__device__ inline Bounds bounds_of(const float* t) {
    return Bounds{t[0], t[1], t[2], t[3], t[4], t[5], t[6], t[7]};
}

template <int NC>
__global__ __launch_bounds__(64 * kWaves) void variant_quantize_kernel(VariantArgs a) {
    constexpr int D = 64 * NC;
    const int lane = threadIdx.x & 63;
    const int64_t vec = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
    if (vec >= (int64_t)a.n * a.H) return;   // uniform per wave
    const VariantInfo vi = a.info;
    const int mid = vi.n_in;
    const Bounds b = bounds_of(a.thr8 + (vec % a.H) * 8);

    float mag[NC];
    int grp[NC];
    bool side[NC];
    float mn[kMaxGroups], mx[kMaxGroups];
#pragma unroll
    for (int k = 0; k < kMaxGroups; ++k) {
        mn[k] = INFINITY;
        mx[k] = -INFINITY;
    }
    const uint16_t* x = a.x + vec * D;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const float xf = h2f(x[64 * c + lane]);
        // from the outside in; a value on a boundary stays on its inner side (Eq. 1)
        const bool ob = vi.n_out == 2 && (xf < b.lo_ob || xf > b.hi_ob);
        const bool oa = !ob && (xf < b.lo_oa || xf > b.hi_oa);
        const bool md = !ob && !oa && (vi.n_in == 0 || xf < b.lo_ia || xf > b.hi_ia);
        const bool md_shift = md && vi.n_in > 0;
        const bool ia = !ob && !oa && !md && vi.n_in == 2 && (xf < b.lo_ib || xf > b.hi_ib);
        const int g = ob ? mid + 2 : oa ? mid + 1 : md ? mid : ia ? 1 : 0;
        const bool shifted = ob || oa || md_shift || ia;
        const float lo_t = ob ? b.lo_ob : oa ? b.lo_oa : md_shift ? b.lo_ia : b.lo_ib;
        const float hi_t = ob ? b.hi_ob : oa ? b.hi_oa : md_shift ? b.hi_ia : b.hi_ib;
        const bool sd = shifted ? (xf > hi_t) : (xf >= 0.0f);
        const float m = shifted ? fabsf(xf - (sd ? hi_t : lo_t)) : fabsf(xf);
        mag[c] = m;
        grp[c] = g;
        side[c] = sd;
#pragma unroll
        for (int k = 0; k < kMaxGroups; ++k) {
            mn[k] = (g == k) ? fminf(mn[k], m) : mn[k];
            mx[k] = (g == k) ? fmaxf(mx[k], m) : mx[k];
        }
    }

    // Eq. 2 per group over the wave; an empty group gets (0, 0)
    float gmin[kMaxGroups], gsig[kMaxGroups];
    uint16_t meta_bits = 0;
#pragma unroll
    for (int k = 0; k < kMaxGroups; ++k) {
        gmin[k] = 0.0f;
        gsig[k] = 0.0f;
        if (k < vi.groups) {
            float lo = wave_reduce(mn[k], INFINITY, [](float p, float q) { return fminf(p, q); });
            float hi = wave_reduce(mx[k], -INFINITY, [](float p, float q) { return fmaxf(p, q); });
            if (!(hi >= lo)) {
                lo = 0.0f;
                hi = 0.0f;
            }
            const float levels = (float)((1 << (k == mid ? 3 : vi.out_bits)) - 1);
            const float range = hi - lo;
            gmin[k] = lo;
            gsig[k] = (range == 0.0f) ? 0.0f : levels / range;
            if (lane == 2 * k) meta_bits = f2h(lo);
            if (lane == 2 * k + 1) meta_bits = f2h(range / levels);
        }
    }
    if (lane < 2 * vi.groups) a.meta[vec * 2 * vi.groups + lane] = meta_bits;

    // Eq. 3, nibbles and COO entries
    int written = 0;
    uint8_t* coo = a.coo + vec * D * vi.coo_bytes;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int g = grp[c];
        const int levels = (1 << (g == mid ? 3 : vi.out_bits)) - 1;
        float gm = gmin[0], gs = gsig[0];
#pragma unroll
        for (int k = 1; k < kMaxGroups; ++k) {
            gm = (g == k) ? gmin[k] : gm;
            gs = (g == k) ? gsig[k] : gs;
        }
        int code = (int)rintf((mag[c] - gm) * gs);
        code = min(max(code, 0), levels);
        const int u = side[c] ? (levels + 1) + code : levels - code;
        const int partner = __shfl_down(u & 15, 1, 64);
        if ((lane & 1) == 0) a.nib[vec * (D / 2) + 32 * c + (lane >> 1)] = (uint8_t)((u & 15) | (partner << 4));
        const bool outl = g != mid;
        const uint64_t m = __ballot(outl);
        const int rank_in_chunk = __popcll(m & ((1ull << lane) - 1ull));
        if (outl) {
            const uint32_t rank = (uint32_t)(g < mid ? g : g - 1);
            uint32_t e = (rank << 6) | (uint32_t)lane;
            if (vi.out_bits == 4) e |= (uint32_t)(u >> 4) << (6 + vi.rank_bits);
            const int slot = written + rank_in_chunk;
            if (vi.coo_bytes == 2)
                reinterpret_cast<uint16_t*>(coo)[slot] = (uint16_t)e;
            else
                coo[slot] = (uint8_t)e;
        }
        const int cnt = __popcll(m);
        if (lane == 0) a.counts[vec * NC + c] = (uint8_t)cnt;
        written += cnt;
    }
    if (lane == 0) a.n_coo[vec] = written;
}

// Dequantization of a variant encoding (fp32): COO entries are scattered back to their
// lanes through LDS, then each value is the side's boundary plus or minus Min + c * Delta.
template <int NC>
__global__ __launch_bounds__(64 * kWaves) void variant_dequantize_kernel(VariantArgs a) {
    constexpr int D = 64 * NC;
    __shared__ uint16_t s_ent[kWaves][D];
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int64_t vec = (int64_t)blockIdx.x * kWaves + w;
    if (vec >= (int64_t)a.n * a.H) return;   // uniform per wave; no workgroup barrier below
    const VariantInfo vi = a.info;
    const int mid = vi.n_in;
    const Bounds b = bounds_of(a.thr8 + (vec % a.H) * 8);
    const uint8_t* coo = a.coo + vec * D * vi.coo_bytes;

#pragma unroll
    for (int c = 0; c < NC; ++c) s_ent[w][64 * c + lane] = 0xffffu;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    int start = 0;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int cnt = min((int)a.counts[vec * NC + c], 64);
        if (lane < cnt) {
            const int k = start + lane;
            const uint32_t e = vi.coo_bytes == 2 ? reinterpret_cast<const uint16_t*>(coo)[k] : coo[k];
            s_ent[w][64 * c + (e & 63u)] = (uint16_t)e;
        }
        start += cnt;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    const uint16_t* meta = a.meta + vec * 2 * vi.groups;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int j = 64 * c + lane;
        int u = (a.nib[vec * (D / 2) + (j >> 1)] >> (4 * (j & 1))) & 15;
        const uint32_t e = s_ent[w][j];
        int g = mid;
        if (e != 0xffffu) {
            const int rank = (int)((e >> 6) & ((1u << vi.rank_bits) - 1u));
            g = rank < mid ? rank : rank + 1;
            if (vi.out_bits == 4) u |= (int)((e >> (6 + vi.rank_bits)) & 1u) << 4;
        }
        g = min(g, vi.groups - 1);
        const int bits = g == mid ? 3 : vi.out_bits;
        const int half = 1 << bits;
        const int hi = u >> bits;
        const int code = hi ? u - half : half - 1 - u;
        const float m = h2f(meta[2 * g]) + (float)code * h2f(meta[2 * g + 1]);
        float lo_t = 0.0f, hi_t = 0.0f;
        if (g == mid + 2) {
            lo_t = b.lo_ob;
            hi_t = b.hi_ob;
        } else if (g == mid + 1) {
            lo_t = b.lo_oa;
            hi_t = b.hi_oa;
        } else if (g == mid && vi.n_in > 0) {
            lo_t = b.lo_ia;
            hi_t = b.hi_ia;
        } else if (g == 1 && vi.n_in == 2) {
            lo_t = b.lo_ib;
            hi_t = b.hi_ib;
        }
        a.out[vec * D + j] = hi ? hi_t + m : lo_t - m;
    }
}

}  // namespace

hipError_t launch_variant_quantize(const VariantArgs& a, int d, hipStream_t st) {
    const int64_t vecs = (int64_t)a.n * a.H;
    const dim3 grid((unsigned)((vecs + kWaves - 1) / kWaves));
    if (d == 64)
        hipLaunchKernelGGL(variant_quantize_kernel<1>, grid, dim3(64 * kWaves), 0, st, a);
    else if (d == 128)
        hipLaunchKernelGGL(variant_quantize_kernel<2>, grid, dim3(64 * kWaves), 0, st, a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_variant_dequantize(const VariantArgs& a, int d, hipStream_t st) {
    const int64_t vecs = (int64_t)a.n * a.H;
    const dim3 grid((unsigned)((vecs + kWaves - 1) / kWaves));
    if (d == 64)
        hipLaunchKernelGGL(variant_dequantize_kernel<1>, grid, dim3(64 * kWaves), 0, st, a);
    else if (d == 128)
        hipLaunchKernelGGL(variant_dequantize_kernel<2>, grid, dim3(64 * kWaves), 0, st, a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace oaken
