// Batched decode attention over the Oaken-quantized paged cache (Oaken Sec. 2.1;
// dequantization engine of Sec. 5.2).
//
// One workgroup owns (sequence, KV head, range of pages) and all query heads that
// share the KV head.  Two passes over the range: first every key page (scores into
// LDS), then the softmax over the range, then every value page.  Ranges of one
// sequence are merged by a log-sum-exp combine.  Each page record is staged in LDS;
// its COO stream is expanded back to positions (the engine's zero-insert) into a
// per-page class map before the dense nibbles are dequantized.
#include "oaken_internal.h"

#include <hip/hip_fp16.h>

namespace oaken {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxG = 8;            // query heads per KV head
constexpr int kScoreCap = 8192;     // fp32 scores per workgroup (G * tokens in range)

__device__ inline float h2f(uint16_t b) { return __half2float(__ushort_as_half(b)); }

// Dequantized value of one element.  cls = 0 for a middle value, else 1 + (COO >> 6).
__device__ inline float dequant(int nib, int cls, const float* m, float lo_o, float lo_i,
                                float hi_i, float hi_o) {
    if (cls == 0) {
        const int hi = nib >> 3;
        const int c = hi ? nib - 8 : 7 - nib;
        const float mag = m[2] + (float)c * m[3];
        return hi ? hi_i + mag : lo_i - mag;
    }
    const int code = cls - 1;
    const int side = code >> 1, outer = code & 1;
    const int c = side ? nib : 15 - nib;
    const float mag = (outer ? m[4] : m[0]) + (float)c * (outer ? m[5] : m[1]);
    if (outer) return side ? hi_o + mag : lo_o - mag;
    return side ? mag : -mag;
}

template <int D>
__device__ void stage_record(const uint8_t* rec, uint8_t* s_rec, uint8_t (*s_cls)[D],
                             float (*s_meta)[6]) {
    constexpr Layout LY = make_layout(kPage, D);
    constexpr int NC = D / 64;
    const int tid = threadIdx.x;
    for (int i = tid; i < (int)(LY.stride / 16); i += kThreads)
        reinterpret_cast<uint4*>(s_rec)[i] = reinterpret_cast<const uint4*>(rec)[i];
    for (int i = tid; i < kPage * D / 4; i += kThreads)
        reinterpret_cast<uint32_t*>(&s_cls[0][0])[i] = 0u;
    __syncthreads();
    if (tid < kPage * NC) {
        const int t = tid / NC, c = tid % NC;
        int start = 0;
        for (int k = 0; k < tid; ++k) start += s_rec[LY.counts + k];
        const int cnt = min((int)s_rec[LY.counts + tid], kPage * D - start);   // stay inside the record
        for (int k = 0; k < cnt; ++k) {
            const int b = s_rec[LY.sparse + start + k];
            s_cls[t][c * 64 + (b & 63)] = (uint8_t)(1 + (b >> 6));
        }
    }
    if (tid < kPage * 6) {
        const int t = tid / 6, k = tid % 6;
        s_meta[t][k] = h2f(*reinterpret_cast<const uint16_t*>(s_rec + LY.meta + t * 12 + k * 2));
    }
    __syncthreads();
}

__device__ inline float block_reduce(float v, float* s_tmp, bool is_max) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float w = __shfl_xor(v, o, 64);
        v = is_max ? fmaxf(v, w) : v + w;
    }
    if (lane == 0) s_tmp[wave] = v;
    __syncthreads();
    float r = s_tmp[0];
    for (int k = 1; k < kThreads / 64; ++k) r = is_max ? fmaxf(r, s_tmp[k]) : r + s_tmp[k];
    __syncthreads();
    return r;
}

template <int D>
__global__ __launch_bounds__(kThreads) void attn_split_kernel(AttnArgs a) {
    constexpr Layout LY = make_layout(kPage, D);
    constexpr int TQ = kThreads / D;           // token groups in the value pass
    constexpr int TPG = kPage / TQ;            // tokens per group per page
    constexpr int DPART = D / 16;              // dims per thread in the key pass

    extern __shared__ float s_scores[];        // [G][range tokens]
    __shared__ __align__(16) uint8_t s_rec[LY.stride];
    __shared__ uint8_t s_cls[kPage][D];
    __shared__ float s_meta[kPage][6];
    __shared__ float s_q[kMaxG][D];
    __shared__ float s_acc[TQ][kMaxG][D];
    __shared__ float s_tmp[kThreads / 64];

    const AttnTile tile = attn_tile(a);
    const int split = tile.split, h = tile.h, s = tile.s;
    const int G = a.Hq / a.H;
    const int tid = threadIdx.x;
    const int L = max(0, min(a.seq_lens[s], min(a.max_seq_len, a.max_blocks * kPage)));
    const int n_pages = (L + kPage - 1) / kPage;
    // a sliding window hides keys before lo; the ranges start at its first page
    const int lo = (a.window > 0 && L > a.window) ? L - a.window : 0;
    const int p_begin = lo / kPage + split * a.pages_per_split;
    const int p_end = min(n_pages, p_begin + a.pages_per_split);
    const int n_tok = max(0, min(L, p_end * kPage) - p_begin * kPage);
    const int tok_cap = a.pages_per_split * kPage;

    for (int i = tid; i < G * D; i += kThreads) {
        const int g = i / D, j = i % D;
        s_q[g][j] = h2f(a.q[((int64_t)s * a.Hq + h * G + g) * D + j]);
    }
    const float* tk = a.thr + (h * 2 + 0) * 4;
    const float* tv = a.thr + (h * 2 + 1) * 4;
    __syncthreads();

    // ---- pass 1: scores ---------------------------------------------------------
    for (int p = p_begin; p < p_end; ++p) {
        const int blk = a.block_table[(int64_t)s * a.max_blocks + p];
        const bool ok = blk >= 0 && blk < a.num_blocks;
        if (ok) stage_record<D>(a.pool + (((int64_t)blk * a.H + h) * 2 + 0) * a.stride, s_rec, s_cls, s_meta);
        const int t = tid / 16, part = tid % 16;
        float acc[kMaxG];
        for (int g = 0; g < kMaxG; ++g) acc[g] = 0.0f;
        if (ok) {
            for (int k = 0; k < DPART; ++k) {
                const int j = part * DPART + k;
                const int byte = s_rec[LY.dense + t * (D / 2) + j / 2];
                const int nib = (j & 1) ? (byte >> 4) : (byte & 15);
                const float v = dequant(nib, s_cls[t][j], s_meta[t], tk[0], tk[1], tk[2], tk[3]);
                for (int g = 0; g < G; ++g) acc[g] += s_q[g][j] * v;
            }
        }
        for (int g = 0; g < G; ++g) {
            float v = acc[g];
#pragma unroll
            for (int o = 8; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
            const int tok = (p - p_begin) * kPage + t;
            const bool valid = ok && (p * kPage + t) < L && (p * kPage + t) >= lo;
            if (part == 0) s_scores[g * tok_cap + tok] = valid ? v * a.scale : -INFINITY;
        }
        __syncthreads();
    }

    // ---- softmax over the range --------------------------------------------------
    float m_g[kMaxG], l_g[kMaxG];
    for (int g = 0; g < G; ++g) {
        float mx = -INFINITY;
        for (int i = tid; i < n_tok; i += kThreads) mx = fmaxf(mx, s_scores[g * tok_cap + i]);
        mx = block_reduce(mx, s_tmp, true);
        float sum = 0.0f;
        for (int i = tid; i < n_tok; i += kThreads) {
            const float sc = s_scores[g * tok_cap + i];
            const float pr = (mx == -INFINITY) ? 0.0f : __expf(sc - mx);
            s_scores[g * tok_cap + i] = pr;
            sum += pr;
        }
        sum = block_reduce(sum, s_tmp, false);
        m_g[g] = mx;
        l_g[g] = sum;
    }
    __syncthreads();

    // ---- pass 2: values ----------------------------------------------------------
    const int j = tid % D, tq = tid / D;
    float o[kMaxG];
    for (int g = 0; g < kMaxG; ++g) o[g] = 0.0f;
    for (int p = p_begin; p < p_end; ++p) {
        const int blk = a.block_table[(int64_t)s * a.max_blocks + p];
        const bool ok = blk >= 0 && blk < a.num_blocks;
        if (ok) stage_record<D>(a.pool + (((int64_t)blk * a.H + h) * 2 + 1) * a.stride, s_rec, s_cls, s_meta);
        if (ok) {
            for (int k = 0; k < TPG; ++k) {
                const int t = tq * TPG + k;
                const int tok = (p - p_begin) * kPage + t;
                if (tok >= n_tok) continue;
                const int byte = s_rec[LY.dense + j * (kPage / 2) + t / 2];
                const int nib = (t & 1) ? (byte >> 4) : (byte & 15);
                const float v = dequant(nib, s_cls[t][j], s_meta[t], tv[0], tv[1], tv[2], tv[3]);
                for (int g = 0; g < G; ++g) o[g] += s_scores[g * tok_cap + tok] * v;
            }
        }
        __syncthreads();
    }
    for (int g = 0; g < G; ++g) s_acc[tq][g][j] = o[g];
    __syncthreads();
    if (tq == 0) {
        for (int g = 0; g < G; ++g) {
            float v = 0.0f;
            for (int k = 0; k < TQ; ++k) v += s_acc[k][g][j];
            const int64_t row = (int64_t)s * a.Hq + h * G + g;
            if (a.n_splits == 1) {
                a.out[row * D + j] = (l_g[g] > 0.0f) ? v / l_g[g] : 0.0f;
            } else {
                float* pp = a.partial + (row * a.n_splits + split) * (D + 2);
                pp[j] = v;
                if (j == 0) { pp[D] = m_g[g]; pp[D + 1] = l_g[g]; }
            }
        }
    }
}

// Log-sum-exp merge of the page ranges' partials (m, l, o) of one (sequence, query head)
// row.  NW waves share the row's ranges (wave w takes ranges w, w + NW, ...), each lane
// D / 64 channels, with a running maximum (the sums are rescaled when it grows), unrolled
// so that several ranges' loads are in flight together; ranges with l = 0 are skipped.
// Decode rows (seq_lens given) read only the ranges that hold keys of their sequence:
// those starting before its last page (the others are empty by construction), so a batch
// of mixed lengths reads no partials of the empty ranges.  The waves' (M, den, num) then
// meet in LDS.
template <int D, int NW>
__global__ __launch_bounds__(64 * NW) void attn_combine_kernel(AttnArgs a) {
    constexpr int V = D / 64;
    const int64_t row = blockIdx.x;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const float* pp = a.partial + row * a.n_splits * (D + 2);
    int n_used = a.n_splits;
    if (a.seq_lens) {
        // the page ranges of the attention kernels: range k starts at page lo / P + k * pps
        const int s = (int)(row / a.Hq);
        const int L = max(0, min(a.seq_lens[s], min(a.max_seq_len, a.max_blocks * kPage)));
        const int n_pages = (L + kPage - 1) / kPage;
        const int lo = (a.window > 0 && L > a.window) ? L - a.window : 0;
        n_used = min(a.n_splits, (n_pages - lo / kPage + a.pages_per_split - 1) / a.pages_per_split);
    }
    float M = -INFINITY, den = 0.0f, num[V];
#pragma unroll
    for (int v = 0; v < V; ++v) num[v] = 0.0f;
#pragma unroll 4
    for (int k = w; k < n_used; k += NW) {
        const float* pk = pp + (int64_t)k * (D + 2);
        const float m = pk[D], l = pk[D + 1];
        float o[V];
        if constexpr (V == 2) {
            const float2 t = *reinterpret_cast<const float2*>(pk + 2 * lane);   // (D + 2) * 4 is a multiple of 8
            o[0] = t.x;
            o[1] = t.y;
        } else {
            o[0] = pk[lane];
        }
        if (l > 0.0f) {
            const float Mn = fmaxf(M, m);
            const float r = __expf(M - Mn), e = __expf(m - Mn);
#pragma unroll
            for (int v = 0; v < V; ++v) num[v] = fmaf(num[v], r, e * o[v]);
            den = fmaf(den, r, e * l);
            M = Mn;
        }
    }
    if constexpr (NW > 1) {
        __shared__ float s_md[NW][2];
        __shared__ float s_num[NW][D];
        if (lane == 0) {
            s_md[w][0] = M;
            s_md[w][1] = den;
        }
#pragma unroll
        for (int v = 0; v < V; ++v) s_num[w][V * lane + v] = num[v];
        __syncthreads();
        if (w != 0) return;
        float Mx = -INFINITY;
#pragma unroll
        for (int x = 0; x < NW; ++x)
            if (s_md[x][1] > 0.0f) Mx = fmaxf(Mx, s_md[x][0]);
        den = 0.0f;
#pragma unroll
        for (int v = 0; v < V; ++v) num[v] = 0.0f;
#pragma unroll
        for (int x = 0; x < NW; ++x) {
            const float r = s_md[x][1] > 0.0f ? __expf(s_md[x][0] - Mx) : 0.0f;
            den = fmaf(s_md[x][1], r, den);
#pragma unroll
            for (int v = 0; v < V; ++v) num[v] = fmaf(s_num[x][V * lane + v], r, num[v]);
        }
    }
#pragma unroll
    for (int v = 0; v < V; ++v) a.out[row * D + V * lane + v] = (den > 0.0f) ? num[v] / den : 0.0f;
}

}  // namespace

SplitPlan plan_splits(int32_t n_seqs, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                      int32_t max_seq_len) {
    const int G = n_q_heads / n_kv_heads;
    const bool mfma = mfma_attention_supported(head_dim, G);
    const int max_pages = (max_seq_len + kPage - 1) / kPage;
    const int64_t units = (int64_t)n_seqs * n_kv_heads * (mfma ? G / mfma_wave_heads(G) : 1);
    const int64_t target = 4096;   // workgroups that keep 256 CUs busy
    int want = (int)((target + units - 1) / units);
    int pps = (max_pages + want - 1) / want;
    pps = max(pps, 8);
    if (mfma)
        pps = min(pps, mfma_score_cap(mfma_wave_heads(G)) / kPage);
    else
        pps = min(pps, kScoreCap / (kPage * G));
    pps = max(pps, 1);
    SplitPlan sp;
    sp.pages_per_split = pps;
    sp.n_splits = (max_pages + pps - 1) / pps;
    return sp;
}

// Waves per row of the combine: about eight ranges per wave, at most eight waves.
template <int D>
hipError_t launch_combine_d(const AttnArgs& a, hipStream_t st) {
    const dim3 grid((uint32_t)((int64_t)a.n_seqs * a.Hq));
    if (a.n_splits <= 8)
        hipLaunchKernelGGL((attn_combine_kernel<D, 1>), grid, dim3(64), 0, st, a);
    else if (a.n_splits <= 16)
        hipLaunchKernelGGL((attn_combine_kernel<D, 2>), grid, dim3(128), 0, st, a);
    else if (a.n_splits <= 32)
        hipLaunchKernelGGL((attn_combine_kernel<D, 4>), grid, dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL((attn_combine_kernel<D, 8>), grid, dim3(512), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_combine(const AttnArgs& a, int d, hipStream_t st) {
    if (d == 64) return launch_combine_d<64>(a, st);
    if (d == 128) return launch_combine_d<128>(a, st);
    return hipErrorInvalidValue;
}

hipError_t launch_attention(const AttnArgs& args, int d, hipStream_t st) {
    AttnArgs a = args;
    const int G = a.Hq / a.H;
    if (G < 1 || G > kMaxG) return hipErrorInvalidValue;
    const bool mfma = mfma_attention_supported(d, G);
    a.wave_heads = mfma ? mfma_wave_heads(G) : G;
    a.head_parts = G / a.wave_heads;
    const size_t shm = (size_t)G * a.pages_per_split * kPage * sizeof(float);
    const uint32_t grid = attn_grid(a);
    if (grid == 0) return hipErrorInvalidValue;
    if (mfma) {
        hipError_t e = launch_attention_mfma(a, st);
        if (e != hipSuccess || a.n_splits == 1) return e;
        return launch_combine(a, d, st);
    }
    if (d == 64) {
        hipLaunchKernelGGL(attn_split_kernel<64>, dim3(grid), dim3(kThreads), shm, st, a);
    } else if (d == 128) {
        hipLaunchKernelGGL(attn_split_kernel<128>, dim3(grid), dim3(kThreads), shm, st, a);
    } else {
        return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.n_splits == 1) return e;
    return launch_combine(a, d, st);
}

}  // namespace oaken
