// Decode attention over the Oaken-quantized cache on CDNA4 int8 matrix cores
// (head_dim 128, 1, 2 or 4 query heads per KV head).
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
// * Inner and outer values (the COO stream) are corrected afterwards: each entry
//   adds its true value minus the middle reading of its nibble.  One lane walks the
//   entries of one (token, 64-value chunk) bucket, with a per-token table of the
//   eight (group, side, h) offsets in LDS.
//
// One wave owns (sequence, KV head, page range).  Pass 1 streams the key pages and
// leaves scores in LDS, then the range's softmax, then pass 2 streams the value
// pages.  Pages are handled in groups of eight: the group's record heads (counts and
// scales) arrive first, so every sparse offset is known before its bytes are loaded.
#include "oaken_internal.h"

#include <hip/hip_fp16.h>

namespace oaken {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int D = 128;
constexpr int P = kPage;
constexpr Layout LY = make_layout(P, D);   // counts 0, meta 32, dense 224, sparse 1248
constexpr int HB = 224;                    // counts + meta bytes at the start of a record
constexpr int GRP = 8;                     // pages per group
constexpr int KROW = 80;                   // LDS stride of a key token's 64 dense bytes
constexpr int SPCAP = P * D;               // sparse capacity of one record

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

__device__ __forceinline__ v4i mfma(v4i a, v4i b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// Value of four base-256 limbs.
__device__ __forceinline__ float limbs(v4i c) {
    return fmaf(fmaf(fmaf((float)c[3], 256.f, (float)c[2]), 256.f, (float)c[1]), 256.f, (float)c[0]);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ __forceinline__ int wave_max_i(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
    return v;
}

// Fixed-point shift so that |x| * 2^shift < 2^22 for every |x| <= mx.
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

__device__ __forceinline__ Tok token_consts(const uint8_t* meta, const float* th) {
    const uint32_t w0 = *reinterpret_cast<const uint32_t*>(meta);
    const uint32_t w1 = *reinterpret_cast<const uint32_t*>(meta + 4);
    const uint32_t w2 = *reinterpret_cast<const uint32_t*>(meta + 8);
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

// Offsets (true value minus middle reading) indexed by ((COO >> 6) << 1) | h, and the
// slope difference per nibble step: delta = tab.x + n * tab.y.
__device__ __forceinline__ void write_table(float2* tab, const Tok& T) {
    tab[0] = make_float2(T.b_il - T.base, T.kd_i);
    tab[1] = make_float2(T.b_il - T.base - T.gp, T.kd_i);
    tab[2] = make_float2(T.b_ol - T.base, T.kd_o);
    tab[3] = make_float2(T.b_ol - T.base - T.gp, T.kd_o);
    tab[4] = make_float2(T.b_ih - T.base, T.kd_i);
    tab[5] = make_float2(T.b_ih - T.base - T.gp, T.kd_i);
    tab[6] = make_float2(T.b_oh - T.base, T.kd_o);
    tab[7] = make_float2(T.b_oh - T.base - T.gp, T.kd_o);
}

__device__ __forceinline__ uint4 ld16(const uint8_t* p) {
    return *reinterpret_cast<const uint4*>(p);
}

template <int G>
struct Smem {
    float q[G][D];
    int qi[G][D];
    float qsum[G];
    int qshift[G];
    int vshift[G];
    float pbase[G];
    float m[G], l[G];
    __align__(16) uint8_t head[GRP][HB];
    int start[GRP][P + 1];                  // sparse start of each valid slot; [P] = total
    __align__(16) uint8_t dense[2][P * KROW];
    __align__(16) uint8_t sparse[2][SPCAP];
    __align__(16) float2 tab[64][8];
    __align__(16) float2 cgf[G][GRP * P];   // p*Delta, p*Gp of the group's tokens
    int2 cg[G][GRP * P];                    // the same in fixed point
    __align__(16) uint32_t at[G][4][4][4];  // value-pass A operand [head][limb][k-group][feature]
    float oc[G][D];                         // value corrections
};

template <int G>
__global__ __launch_bounds__(64) void attn_mfma_kernel(AttnArgs a) {
    constexpr int NRS = (G + 1) / 2;        // key-pass MFMA row sets (8 rows per head)
    __shared__ Smem<G> S;
    extern __shared__ float sc[];           // [G][cap]: scores, then probabilities

    const int lane = threadIdx.x;
    const int split = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
    const int L = max(0, min(a.seq_lens[s], min(a.max_seq_len, a.max_blocks * P)));
    const int n_pages = (L + P - 1) / P;
    const int p_begin = split * a.pages_per_split;
    const int p_end = min(n_pages, p_begin + a.pages_per_split);
    const int cap = a.pages_per_split * P;
    const int n_tok = max(0, min(L, p_end * P) - p_begin * P);
    const int32_t* btab = a.block_table + (int64_t)s * a.max_blocks;

    float tk[4], tv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        tk[i] = fin(a.thr[(h * 2 + 0) * 4 + i]);
        tv[i] = fin(a.thr[(h * 2 + 1) * 4 + i]);
    }
    auto record = [&](int page, int which) -> const uint8_t* {
        const int blk = btab[page];
        if (blk < 0 || blk >= a.num_blocks) return nullptr;
        return a.pool + (((int64_t)blk * a.H + h) * 2 + which) * a.stride;
    };
    auto valid_slots = [&](int page) -> int { return max(0, min(P, L - page * P)); };

    // ---- query in fp32 and in fixed point -----------------------------------------
#pragma unroll
    for (int hd = 0; hd < G; ++hd) {
        const uint16_t* qp = a.q + ((int64_t)s * a.Hq + h * G + hd) * D;
        const float x0 = h2f(qp[lane]), x1 = h2f(qp[lane + 64]);
        S.q[hd][lane] = x0;
        S.q[hd][lane + 64] = x1;
        const float mx = wave_max(fmaxf(fabsf(x0), fabsf(x1)));
        const float sum = wave_sum(x0 + x1);
        const int sh = fix_shift(mx);
        S.qi[hd][lane] = (int)rintf(ldexpf(x0, sh));
        S.qi[hd][lane + 64] = (int)rintf(ldexpf(x1, sh));
        if (lane == 0) {
            S.qsum[hd] = sum;
            S.qshift[hd] = sh;
        }
    }
    __syncthreads();

    // Key-pass A operand: row = 8*(head%2) + 4*type + limb, type 0 -> sum q u, 1 -> sum q h.
    // Byte (4f + b) of k-group g4 in MFMA m pairs with feature f of dense byte 16*g4+4*m+b.
    v4i afk[NRS][4];
    {
        const int row = lane & 15, g4 = lane >> 4, type = (row >> 2) & 1, r = row & 3;
#pragma unroll
        for (int rs = 0; rs < NRS; ++rs) {
            const int hd = rs * 2 + (row >> 3);
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                uint32_t f0 = 0, f1 = 0, f2 = 0, f3 = 0;
                if (hd < G) {
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        const int pr = g4 * 16 + m * 4 + b;
                        const int qe = S.qi[hd][2 * pr], qo = S.qi[hd][2 * pr + 1];
                        const int w0 = type ? 0 : 8 * qo;
                        const int w1 = type ? 0 : 128 * qe - 8 * qo;
                        const int w2 = type ? -qo : -16 * qo;
                        const int w3 = type ? 16 * qe + qo : 16 * qo;
                        f0 |= byte_of(enc(w0), r) << (8 * b);
                        f1 |= byte_of(enc(w1), r) << (8 * b);
                        f2 |= byte_of(enc(w2), r) << (8 * b);
                        f3 |= byte_of(enc(w3), r) << (8 * b);
                    }
                }
                afk[rs][m][0] = (int)f0;
                afk[rs][m][1] = (int)f1;
                afk[rs][m][2] = (int)f2;
                afk[rs][m][3] = (int)f3;
            }
        }
    }

    // Loads the heads of a group and the sparse start offsets of its valid slots.
    auto load_group_heads = [&](int g0, int npg, int which) {
        for (int c = lane; c < GRP * 14; c += 64) {
            const int pg = c / 14, off = (c % 14) * 16;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (pg < npg) {
                const uint8_t* rec = record(g0 + pg, which);
                if (rec) v = ld16(rec + off);
            }
            *reinterpret_cast<uint4*>(&S.head[pg][off]) = v;
        }
        __syncthreads();
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int pg = half * 4 + (lane >> 4), t = lane & 15;
            const bool ok = pg < npg && record(g0 + pg, which) != nullptr && t < valid_slots(g0 + pg);
            const int tot = ok ? (int)S.head[pg][2 * t] + (int)S.head[pg][2 * t + 1] : 0;
            int incl = tot;
#pragma unroll
            for (int d = 1; d < 16; d <<= 1) {
                const int y = __shfl_up(incl, d, 16);
                if (t >= d) incl += y;
            }
            S.start[pg][t] = incl - tot;
            if (t == 15) S.start[pg][P] = min(incl, SPCAP);
        }
        __syncthreads();
    };
    // Copies the used sparse bytes of one page into LDS buffer k2.
    auto load_sparse = [&](int g0, int pg, int npg, int which, int k2) {
        if (pg >= npg) return;
        const uint8_t* rec = record(g0 + pg, which);
        if (!rec) return;
        const int nch = (S.start[pg][P] + 15) >> 4;
        for (int c = lane; c < nch; c += 64)
            *reinterpret_cast<uint4*>(&S.sparse[k2][16 * c]) = ld16(rec + LY.sparse + 16 * c);
    };

    // ---- pass 1: keys -------------------------------------------------------------
    for (int g0 = p_begin; g0 < p_end; g0 += GRP) {
        const int npg = min(GRP, p_end - g0);
        load_group_heads(g0, npg, 0);
        uint4 dreg[GRP];
#pragma unroll
        for (int pg = 0; pg < GRP; ++pg) {
            dreg[pg] = make_uint4(0, 0, 0, 0);
            if (pg < npg) {
                const uint8_t* rec = record(g0 + pg, 0);
                if (rec) dreg[pg] = ld16(rec + LY.dense + (lane & 15) * 64 + (lane >> 4) * 16);
            }
        }
#pragma unroll
        for (int pp = 0; pp < GRP; pp += 2) {
            if (pp >= npg) break;
            load_sparse(g0, pp, npg, 0, 0);
            load_sparse(g0, pp + 1, npg, 0, 1);
            *reinterpret_cast<uint4*>(&S.dense[0][(lane & 15) * KROW + (lane >> 4) * 16]) = dreg[pp];
            *reinterpret_cast<uint4*>(&S.dense[1][(lane & 15) * KROW + (lane >> 4) * 16]) = dreg[pp + 1];
            // dense part on the matrix cores
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                const int pg = pp + k2;
                const uint4 dv = dreg[pg];
                v4i acc[NRS];
#pragma unroll
                for (int rs = 0; rs < NRS; ++rs) acc[rs] = v4i{0, 0, 0, 0};
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const uint32_t dw = m == 0 ? dv.x : m == 1 ? dv.y : m == 2 ? dv.z : dv.w;
                    const v4i B = features(dw);
#pragma unroll
                    for (int rs = 0; rs < NRS; ++rs) acc[rs] = mfma(afk[rs][m], B, acc[rs]);
                }
                const int t = lane & 15, grp4 = lane >> 4;
                const bool pv = pg < npg && record(g0 + pg, 0) != nullptr;
                const int nval = pv ? valid_slots(g0 + pg) : 0;
                const Tok T = token_consts(&S.head[pg][LY.meta + 12 * t], tk);
                const int tok = (g0 + pg - p_begin) * P + t;
#pragma unroll
                for (int rs = 0; rs < NRS; ++rs) {
                    const float v = limbs(acc[rs]);
                    const float o = __shfl_xor(v, 16, 64);
                    const int hd = rs * 2 + (grp4 >> 1);
                    if ((grp4 & 1) == 0 && hd < G && pg < npg) {
                        const int e = S.qshift[hd] + 7;
                        const float dot = T.base * S.qsum[hd] + T.dm * ldexpf(v, -e) + T.gp * ldexpf(o, -e);
                        sc[hd * cap + tok] = (t < nval) ? a.scale * dot : -INFINITY;
                    }
                }
            }
            __syncthreads();
            // sparse part: lane = (page of pair, chunk, token)
            {
                const int k2 = lane >> 5, c = (lane >> 4) & 1, t = lane & 15;
                const int pg = pp + k2;
                const bool pv = pg < npg && record(g0 + pg, 0) != nullptr;
                const bool vt = pv && t < valid_slots(g0 + pg);
                const int c0 = vt ? (int)S.head[pg][2 * t] : 0;
                const int c1 = vt ? (int)S.head[pg][2 * t + 1] : 0;
                const int st = (vt ? S.start[pg][t] : 0) + (c ? c0 : 0);
                const int cnt = max(0, min(c ? c1 : c0, SPCAP - st));
                if (vt) write_table(S.tab[lane], token_consts(&S.head[pg][LY.meta + 12 * t], tk));
                const int maxc = wave_max_i(cnt);
                const uint8_t* spp = &S.sparse[k2][st];
                const uint8_t* drow = &S.dense[k2][t * KROW + c * 32];
                float corr[G];
#pragma unroll
                for (int hd = 0; hd < G; ++hd) corr[hd] = 0.0f;
                for (int k = 0; k < maxc; ++k) {
                    if (k < cnt) {
                        const uint32_t b = spp[k];
                        const uint32_t dw = *reinterpret_cast<const uint32_t*>(drow + ((b >> 1) & 0x1cu));
                        const uint32_t n = (dw >> ((b & 7u) << 2)) & 15u;
                        const float2 kv = S.tab[lane][((b >> 6) << 1) | (n >> 3)];
                        const float delta = fmaf((float)n, kv.y, kv.x);
                        const int j = c * 64 + (int)(b & 63u);
#pragma unroll
                        for (int hd = 0; hd < G; ++hd) corr[hd] = fmaf(S.q[hd][j], delta, corr[hd]);
                    }
                }
#pragma unroll
                for (int hd = 0; hd < G; ++hd) {
                    const float o = corr[hd] + __shfl_xor(corr[hd], 16, 64);
                    if (c == 0 && vt) sc[hd * cap + (g0 + pg - p_begin) * P + t] += a.scale * o;
                }
            }
            __syncthreads();
        }
    }

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
        S.oc[hd][lane] = 0.0f;
        S.oc[hd][lane + 64] = 0.0f;
    }
    __syncthreads();

    // ---- pass 2: values ------------------------------------------------------------
    const int hq = lane >> 4;               // output lane owns (head hq, dim 16*nt + (lane&15))
    float oacc[8];
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) oacc[nt] = 0.0f;
    float pb[G];
#pragma unroll
    for (int hd = 0; hd < G; ++hd) pb[hd] = 0.0f;

    for (int g0 = p_begin; g0 < p_end; g0 += GRP) {
        const int npg = min(GRP, p_end - g0);
        load_group_heads(g0, npg, 1);
        uint4 dreg[GRP];
#pragma unroll
        for (int pg = 0; pg < GRP; ++pg) {
            dreg[pg] = make_uint4(0, 0, 0, 0);
            if (pg < npg) {
                const uint8_t* rec = record(g0 + pg, 1);
                if (rec) dreg[pg] = ld16(rec + LY.dense + lane * 16);
            }
        }
        // fixed-point coefficients p*Delta, p*Gp of the group's tokens, one shift per head
#pragma unroll
        for (int hd = 0; hd < G; ++hd) {
            float mx = 0.0f;
            for (int tg = lane; tg < GRP * P; tg += 64) {
                const int pg = tg >> 4, t = tg & 15;
                const bool vt = pg < npg && record(g0 + pg, 1) != nullptr && t < valid_slots(g0 + pg);
                float cx = 0.0f, gx = 0.0f;
                if (vt) {
                    const float p = sc[hd * cap + (g0 + pg - p_begin) * P + t];
                    const Tok T = token_consts(&S.head[pg][LY.meta + 12 * t], tv);
                    cx = p * T.dm;
                    gx = p * T.gp;
                    pb[hd] = fmaf(p, T.base, pb[hd]);
                }
                S.cgf[hd][tg] = make_float2(cx, gx);
                mx = fmaxf(mx, fmaxf(fabsf(cx), fabsf(gx)));
            }
            const int sh = fix_shift(wave_max(mx));
            for (int tg = lane; tg < GRP * P; tg += 64) {
                const float2 f = S.cgf[hd][tg];
                S.cg[hd][tg] = make_int2((int)rintf(ldexpf(f.x, sh)), (int)rintf(ldexpf(f.y, sh)));
            }
            if (lane == 0) S.vshift[hd] = sh;
        }
        __syncthreads();

        v4i gacc[8];
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) gacc[nt] = v4i{0, 0, 0, 0};
#pragma unroll
        for (int pp = 0; pp < GRP; pp += 2) {
            if (pp >= npg) break;
            load_sparse(g0, pp, npg, 1, 0);
            load_sparse(g0, pp + 1, npg, 1, 1);
            *reinterpret_cast<uint4*>(&S.dense[0][lane * 16]) = dreg[pp];
            *reinterpret_cast<uint4*>(&S.dense[1][lane * 16]) = dreg[pp + 1];
            // A operand: lane = (limb r, feature f, k-group g4); token pair 4*g4 + b
            {
                const int r = lane & 3, f = (lane >> 2) & 3, g4 = lane >> 4;
                const int al = f == 1 ? 128 : 0;
                const int be = f == 0 ? 8 : f == 1 ? -8 : f == 2 ? -16 : 16;
                const int ga = f == 3 ? 16 : 0;
                const int de = f == 2 ? -1 : f == 3 ? 1 : 0;
#pragma unroll
                for (int hd = 0; hd < G; ++hd) {
                    uint32_t dw = 0;
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        const int te = pp * P + 2 * (g4 * 4 + b);
                        const int2 e = S.cg[hd][te], o = S.cg[hd][te + 1];
                        const int w = al * e.x + be * o.x + ga * e.y + de * o.y;
                        dw |= byte_of(enc(w), r) << (8 * b);
                    }
                    S.at[hd][r][g4][f] = dw;
                }
            }
            __syncthreads();
            {
                const int row = lane & 15, hdr = row >> 2, g4 = lane >> 4;
                v4i av = v4i{0, 0, 0, 0};
                if (hdr < G) av = *reinterpret_cast<const v4i*>(&S.at[hdr][row & 3][g4][0]);
#pragma unroll
                for (int nt = 0; nt < 8; ++nt) {
                    const int j = nt * 16 + (lane & 15);
                    const uint32_t dw =
                        *reinterpret_cast<const uint32_t*>(&S.dense[g4 >> 1][j * 8 + (g4 & 1) * 4]);
                    gacc[nt] = mfma(av, features(dw), gacc[nt]);
                }
            }
            // sparse part: lane = (page of pair, chunk, token)
            {
                const int k2 = lane >> 5, c = (lane >> 4) & 1, t = lane & 15;
                const int pg = pp + k2;
                const bool pv = pg < npg && record(g0 + pg, 1) != nullptr;
                const bool vt = pv && t < valid_slots(g0 + pg);
                const int c0 = vt ? (int)S.head[pg][2 * t] : 0;
                const int c1 = vt ? (int)S.head[pg][2 * t + 1] : 0;
                const int st = (vt ? S.start[pg][t] : 0) + (c ? c0 : 0);
                const int cnt = max(0, min(c ? c1 : c0, SPCAP - st));
                float pt[G];
#pragma unroll
                for (int hd = 0; hd < G; ++hd)
                    pt[hd] = vt ? sc[hd * cap + (g0 + pg - p_begin) * P + t] : 0.0f;
                if (vt) write_table(S.tab[lane], token_consts(&S.head[pg][LY.meta + 12 * t], tv));
                const int maxc = wave_max_i(cnt);
                const uint8_t* spp = &S.sparse[k2][st];
                const uint8_t* dcol = &S.dense[k2][(t >> 3) * 4];
                const int shift = (t & 7) * 4;
                for (int k = 0; k < maxc; ++k) {
                    if (k < cnt) {
                        const uint32_t b = spp[k];
                        const int j = c * 64 + (int)(b & 63u);
                        const uint32_t dw = *reinterpret_cast<const uint32_t*>(dcol + j * 8);
                        const uint32_t n = (dw >> shift) & 15u;
                        const float2 kv = S.tab[lane][((b >> 6) << 1) | (n >> 3)];
                        const float delta = fmaf((float)n, kv.y, kv.x);
#pragma unroll
                        for (int hd = 0; hd < G; ++hd) atomicAdd(&S.oc[hd][j], pt[hd] * delta);
                    }
                }
            }
            __syncthreads();
        }
        // fold the group's integer sums into the fp32 outputs
        if (hq < G) {
            const int e = S.vshift[hq] + 7;
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) oacc[nt] += ldexpf(limbs(gacc[nt]), -e);
        }
        __syncthreads();
    }

#pragma unroll
    for (int hd = 0; hd < G; ++hd) {
        const float v = wave_sum(pb[hd]);
        if (lane == 0) S.pbase[hd] = v;
    }
    __syncthreads();
    if (hq < G) {
        const int64_t row = (int64_t)s * a.Hq + h * G + hq;
        const float l = S.l[hq];
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) {
            const int j = nt * 16 + (lane & 15);
            const float o = S.pbase[hq] + oacc[nt] + S.oc[hq][j];
            if (a.n_splits == 1) {
                a.out[row * D + j] = (l > 0.0f) ? o / l : 0.0f;
            } else {
                float* pp = a.partial + (row * a.n_splits + split) * (D + 2);
                pp[j] = o;
                if (j == 0) {
                    pp[D] = S.m[hq];
                    pp[D + 1] = l;
                }
            }
        }
    }
}

}  // namespace

bool mfma_attention_supported(int d, int G) { return d == D && (G == 1 || G == 2 || G == 4); }

int mfma_score_cap() { return 2048; }

hipError_t launch_attention_mfma(const AttnArgs& a, hipStream_t st) {
    const int G = a.Hq / a.H;
    const size_t shm = (size_t)G * a.pages_per_split * P * sizeof(float);
    dim3 grid(a.n_splits, a.H, a.n_seqs);
    if (G == 1)
        hipLaunchKernelGGL(attn_mfma_kernel<1>, grid, dim3(64), shm, st, a);
    else if (G == 2)
        hipLaunchKernelGGL(attn_mfma_kernel<2>, grid, dim3(64), shm, st, a);
    else if (G == 4)
        hipLaunchKernelGGL(attn_mfma_kernel<4>, grid, dim3(64), shm, st, a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace oaken
