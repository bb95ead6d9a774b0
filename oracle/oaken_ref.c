/*
 * oaken_ref.c -- CPU oracle for Oaken's KV-cache quantizer and decode attention
 * (Kim et al., "Oaken: Fast and Efficient LLM Serving with Online-Offline Hybrid
 * KV Cache Quantization", ISCA 2025).
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load this library.  It shares no
 * source, header, table or helper with the HIP library; the page-record layout
 * is re-derived here from its written definition.
 *
 * Precision: the quantizer follows the paper's Eq. 1-4 in IEEE fp32 (one
 * rounding per operation, no fused multiply-add, round-half-to-even), because
 * the codes it produces are compared bit for bit.  Dequantized values and the
 * attention itself are computed in fp64 from the stored fp16 metadata and the
 * fp32 thresholds: that is the plain definition of softmax(q K^T * scale) V
 * over the dequantized cache.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fopenmp -shared -fPIC
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { REF_INNER = 0, REF_MIDDLE = 1, REF_OUTER = 2 };

/* ------------------------------------------------------------------------ */
/* IEEE binary16 <-> binary32, written out from the format definition.       */
/* ------------------------------------------------------------------------ */

float oaken_ref_half_to_float(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int exp = (h >> 10) & 0x1f;
    int man = h & 0x3ff;
    float v;
    if (exp == 0)
        v = ldexpf((float)man, -24);              /* zero or subnormal */
    else if (exp == 31)
        v = man ? NAN : INFINITY;
    else
        v = ldexpf((float)(man | 0x400), exp - 25);
    return sign ? -v : v;
}

/* Round-to-nearest-even conversion; overflow goes to infinity. */
uint16_t oaken_ref_float_to_half(float f)
{
    uint16_t sign = signbit(f) ? 0x8000 : 0;
    if (isnan(f)) return 0x7e00;
    double a = fabs((double)f);
    if (isinf(f) || a >= 65520.0) return sign | 0x7c00;
    if (a < ldexp(1.0, -14)) {                    /* subnormal range */
        double q = nearbyint(a * ldexp(1.0, 24)); /* exact scaling */
        return sign | (uint16_t)q;                /* q == 1024 is the smallest normal */
    }
    int e2;
    frexp(a, &e2);                                /* a in [2^(e2-1), 2^e2) */
    int E = e2 - 1;
    double q = nearbyint(ldexp(a, 10 - E));       /* in [1024, 2048] */
    if (q >= 2048.0) { q = 1024.0; E += 1; }
    return sign | (uint16_t)(((E + 15) << 10) | ((int)q - 1024));
}

/* ------------------------------------------------------------------------ */
/* Page-record layout (one record per physical block, KV head, and K or V).  */
/*   counts : uint8 [P][d/64]  outliers per (slot, 64-element chunk)         */
/*   meta   : fp16  [P][6]     (Min, Delta) of inner, middle, outer group    */
/*   dense  : nibbles, K token-major, V channel-major                        */
/*   sparse : one COO byte per outlier, slot-major, chunk-major, ascending   */
/* Each of meta and dense starts on a 16-byte boundary; sparse follows dense */
/* directly; the record stride is rounded up to 128 bytes.                   */
/* ------------------------------------------------------------------------ */

static int64_t up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

void oaken_ref_layout(int P, int d, int64_t out[5])
{
    int64_t counts = 0;
    int64_t meta = up(counts + (int64_t)P * (d / 64), 16);
    int64_t dense = up(meta + (int64_t)P * 12, 16);
    int64_t sparse = dense + (int64_t)P * d / 2;
    int64_t stride = up(sparse + (int64_t)P * d, 128);
    out[0] = counts; out[1] = meta; out[2] = dense; out[3] = sparse; out[4] = stride;
}

/* Byte offset (within the dense field) and nibble half of element j of slot t. */
static void dense_pos(int which, int P, int d, int t, int j, int64_t* byte, int* high)
{
    if (which == 0) { *byte = (int64_t)t * (d / 2) + j / 2; *high = j & 1; }
    else            { *byte = (int64_t)j * (P / 2) + t / 2; *high = t & 1; }
}

/* ------------------------------------------------------------------------ */
/* Quantizer for one vector of d values (one token, one KV head, K or V).    */
/* ------------------------------------------------------------------------ */

/*
 * Eq. 1 (Sec. 4.3): the four offline thresholds split the vector into the
 * outer, middle and inner groups.  Eq. 4 (Sec. 4.4): outer and middle values
 * are shifted by the threshold on their side before quantization; inner
 * values are not shifted.  Eq. 2-3: each group is min-max quantized with a
 * scale computed online from that vector's own group minimum and maximum.
 * Sec. 4.4 end: middle codes are 4 bits, inner/outer codes are 5 bits; the
 * side ("sign") is the top bit of the code and the group's min-max grid is
 * applied to the shifted magnitudes (3 resp. 4 bits).
 * Sec. 4.5: middle codes live in the dense nibble matrix; an outlier keeps
 * its low 4 code bits in its dense slot, and its COO byte holds the 6-bit
 * index within its 64-element chunk, one group bit (1 = outer) and the sign
 * bit (1 = upper side).
 *
 * Outputs: code[j] = full code (0..15 middle, 0..31 inner/outer), group[j],
 * meta[6] = fp16 bit patterns (Min, Delta) for inner, middle, outer, the
 * per-chunk outlier counts and the COO bytes in emission order.
 */
void oaken_ref_quantize_vector(const uint16_t* x, int d, const float thr[4],
                               uint8_t* code, uint8_t* group, uint16_t meta[6],
                               uint8_t* counts, uint8_t* coo, int* n_coo)
{
    const float lo_o = thr[0], lo_i = thr[1], hi_i = thr[2], hi_o = thr[3];
    float* a = (float*)malloc(sizeof(float) * d);
    uint8_t* side = (uint8_t*)malloc(d);

    for (int j = 0; j < d; ++j) {
        float xf = oaken_ref_half_to_float(x[j]);
        if (xf < lo_o || xf > hi_o) {                 /* G_o */
            group[j] = REF_OUTER;
            side[j] = xf > hi_o;
            a[j] = fabsf(xf - (side[j] ? hi_o : lo_o));
        } else if (xf < lo_i || xf > hi_i) {          /* G_m */
            group[j] = REF_MIDDLE;
            side[j] = xf > hi_i;
            a[j] = fabsf(xf - (side[j] ? hi_i : lo_i));
        } else {                                      /* G_i, not shifted */
            group[j] = REF_INNER;
            side[j] = xf >= 0.0f;
            a[j] = fabsf(xf);
        }
    }

    for (int g = 0; g < 3; ++g) {
        float mn = INFINITY, mx = -INFINITY;
        int any = 0;
        for (int j = 0; j < d; ++j)
            if (group[j] == g) {
                any = 1;
                if (a[j] < mn) mn = a[j];
                if (a[j] > mx) mx = a[j];
            }
        if (!any) { mn = 0.0f; mx = 0.0f; }
        const int bits = (g == REF_MIDDLE) ? 3 : 4;
        const int levels = (1 << bits) - 1;           /* 2^b - 1 */
        const float range = mx - mn;
        const float sigma = (range == 0.0f) ? 0.0f : (float)levels / range;   /* Eq. 2 */
        for (int j = 0; j < d; ++j) {
            if (group[j] != g) continue;
            float shifted = a[j] - mn;
            float scaled = shifted * sigma;
            float r = rintf(scaled);                                           /* Eq. 3 */
            int c = (int)r;
            if (c < 0) c = 0;
            if (c > levels) c = levels;
            code[j] = (uint8_t)(side[j] ? (levels + 1) + c : levels - c);
        }
        meta[2 * g] = oaken_ref_float_to_half(mn);
        meta[2 * g + 1] = oaken_ref_float_to_half(range / (float)levels);
    }

    int n = 0;
    for (int c = 0; c < d / 64; ++c) {
        int cnt = 0;
        for (int j = c * 64; j < c * 64 + 64; ++j) {
            if (group[j] == REF_MIDDLE) continue;
            coo[n++] = (uint8_t)(((code[j] >> 4) << 7) | ((group[j] == REF_OUTER) << 6) | (j & 63));
            ++cnt;
        }
        counts[c] = (uint8_t)cnt;
    }
    *n_coo = n;
    free(a);
    free(side);
}

/* ------------------------------------------------------------------------ */
/* Writing tokens into page records (Sec. 5.2, MMU: per-head pages, tokens    */
/* appended in order so that a page is read back as one burst).              */
/* ------------------------------------------------------------------------ */

static void write_slot(uint8_t* rec, int which, int P, int d, int slot,
                       const uint8_t* code, const uint16_t meta[6],
                       const uint8_t* counts, const uint8_t* coo, int n_coo)
{
    int64_t L[5];
    oaken_ref_layout(P, d, L);
    const int nc = d / 64;
    int64_t start = 0;
    for (int t = 0; t < slot; ++t)
        for (int c = 0; c < nc; ++c) start += rec[L[0] + (int64_t)t * nc + c];
    for (int c = 0; c < nc; ++c) rec[L[0] + (int64_t)slot * nc + c] = counts[c];
    for (int k = 0; k < 6; ++k) {
        rec[L[1] + (int64_t)slot * 12 + 2 * k] = (uint8_t)(meta[k] & 0xff);
        rec[L[1] + (int64_t)slot * 12 + 2 * k + 1] = (uint8_t)(meta[k] >> 8);
    }
    for (int j = 0; j < d; ++j) {
        int64_t byte; int high;
        dense_pos(which, P, d, slot, j, &byte, &high);
        uint8_t nib = code[j] & 15;
        uint8_t* p = rec + L[2] + byte;
        /* writing a low nibble clears the partner nibble; a high nibble keeps it */
        *p = high ? (uint8_t)((*p & 0x0f) | (nib << 4)) : nib;
    }
    memcpy(rec + L[3] + start, coo, (size_t)n_coo);
}

int oaken_ref_quantize_kv(uint8_t* pool, int num_blocks, int P, int H, int d, int64_t stride,
                          const float* thr, const uint16_t* k_new, const uint16_t* v_new,
                          const int32_t* block_table, int max_blocks,
                          const int32_t* start_pos, const int32_t* cu_tokens, int n_seqs)
{
    int bad = 0;
    /* records of different (sequence, KV head) pairs are disjoint; within one record the
       tokens are written in position order */
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int s = 0; s < n_seqs; ++s)
        for (int h = 0; h < H; ++h) {
            uint8_t* code = (uint8_t*)malloc(d);
            uint8_t* group = (uint8_t*)malloc(d);
            uint8_t* coo = (uint8_t*)malloc(d);
            uint8_t counts[16];
            uint16_t meta[6];
            for (int row = cu_tokens[s]; row < cu_tokens[s + 1]; ++row) {
                const int pos = start_pos[s] + (row - cu_tokens[s]);
                const int lb = pos / P, slot = pos % P;
                if (lb >= max_blocks) { bad = 1; break; }
                const int blk = block_table[(int64_t)s * max_blocks + lb];
                if (blk < 0 || blk >= num_blocks) { bad = 1; break; }
                for (int which = 0; which < 2; ++which) {
                    const uint16_t* x = (which ? v_new : k_new) + ((int64_t)row * H + h) * d;
                    int n_coo = 0;
                    oaken_ref_quantize_vector(x, d, thr + (h * 2 + which) * 4, code, group,
                                              meta, counts, coo, &n_coo);
                    uint8_t* rec = pool + (((int64_t)blk * H + h) * 2 + which) * stride;
                    write_slot(rec, which, P, d, slot, code, meta, counts, coo, n_coo);
                }
            }
            free(code); free(group); free(coo);
        }
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Dequantization of one stored slot (Sec. 5.2 dequantization engine: the    */
/* COO stream is zero-inserted back to its positions and merged with the     */
/* dense nibbles).  Result in fp64.                                          */
/* ------------------------------------------------------------------------ */

void oaken_ref_dequantize_slot(const uint8_t* rec, int which, int P, int d, int slot,
                               const float thr[4], double* out, uint8_t* group_out)
{
    int64_t L[5];
    oaken_ref_layout(P, d, L);
    const int nc = d / 64;
    int* u = (int*)malloc(sizeof(int) * d);
    uint8_t* grp = (uint8_t*)malloc(d);
    for (int j = 0; j < d; ++j) {
        int64_t byte; int high;
        dense_pos(which, P, d, slot, j, &byte, &high);
        uint8_t b = rec[L[2] + byte];
        u[j] = high ? (b >> 4) : (b & 15);
        grp[j] = REF_MIDDLE;
    }
    int64_t e = 0;
    for (int t = 0; t < slot; ++t)
        for (int c = 0; c < nc; ++c) e += rec[L[0] + (int64_t)t * nc + c];
    for (int c = 0; c < nc; ++c) {
        int cnt = rec[L[0] + (int64_t)slot * nc + c];
        for (int k = 0; k < cnt; ++k) {
            uint8_t b = rec[L[3] + e++];
            int j = c * 64 + (b & 63);
            grp[j] = (b & 0x40) ? REF_OUTER : REF_INNER;
            u[j] = ((b >> 7) << 4) | u[j];
        }
    }
    double Min[3], Del[3];
    for (int g = 0; g < 3; ++g) {
        uint16_t mb = (uint16_t)(rec[L[1] + (int64_t)slot * 12 + 4 * g] |
                                 (rec[L[1] + (int64_t)slot * 12 + 4 * g + 1] << 8));
        uint16_t db = (uint16_t)(rec[L[1] + (int64_t)slot * 12 + 4 * g + 2] |
                                 (rec[L[1] + (int64_t)slot * 12 + 4 * g + 3] << 8));
        Min[g] = oaken_ref_half_to_float(mb);
        Del[g] = oaken_ref_half_to_float(db);
    }
    const double lo_o = thr[0], lo_i = thr[1], hi_i = thr[2], hi_o = thr[3];
    for (int j = 0; j < d; ++j) {
        const int g = grp[j];
        const int bits = (g == REF_MIDDLE) ? 3 : 4;
        const int half = 1 << bits;
        const int hi = u[j] >> bits;
        const int c = hi ? u[j] - half : half - 1 - u[j];
        const double mag = Min[g] + (double)c * Del[g];
        double v;
        if (g == REF_INNER)       v = hi ? mag : -mag;
        else if (g == REF_MIDDLE) v = hi ? hi_i + mag : lo_i - mag;
        else                      v = hi ? hi_o + mag : lo_o - mag;
        out[j] = v;
        if (group_out) group_out[j] = (uint8_t)g;
    }
    free(u);
    free(grp);
}

/* ------------------------------------------------------------------------ */
/* Decode attention over the dequantized cache (Sec. 2.1: the new query is   */
/* multiplied with every cached key, softmax, then weighted sum of values).  */
/* Query head h reads KV head h / (Hq / H).  fp64 throughout.               */
/* With a sliding window W > 0 (the Mistral/Mixtral models of Sec. 6.1) the  */
/* query at position L-1 sees only keys t with L-W <= t < L; W <= 0 means    */
/* the whole sequence.                                                       */
/* ------------------------------------------------------------------------ */

int oaken_ref_decode_attention(const uint8_t* pool, int num_blocks, int P, int H, int d,
                               int64_t stride, const float* thr, const uint16_t* q, int Hq,
                               const int32_t* block_table, int max_blocks,
                               const int32_t* seq_lens, int n_seqs, int window, float scale,
                               float* out)
{
    if (Hq % H != 0) return -1;
    const int G = Hq / H;
    int bad = 0;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int s = 0; s < n_seqs; ++s)
        for (int h = 0; h < H; ++h) {
            const int Ls = seq_lens[s];
            const int t0 = (window > 0 && Ls > window) ? Ls - window : 0;   /* first key seen */
            double* kv = (double*)malloc(sizeof(double) * d);
            double* sc = (double*)malloc(sizeof(double) * (size_t)Ls * G);
            double* acc = (double*)calloc((size_t)G * d, sizeof(double));
            double* qd = (double*)malloc(sizeof(double) * (size_t)G * d);
            for (int gq = 0; gq < G; ++gq)
                for (int j = 0; j < d; ++j)
                    qd[gq * d + j] = oaken_ref_half_to_float(q[((int64_t)s * Hq + h * G + gq) * d + j]);
            int ok = Ls >= 1 && (Ls + P - 1) / P <= max_blocks;
            for (int t = t0; ok && t < Ls; ++t) {
                int blk = block_table[(int64_t)s * max_blocks + t / P];
                if (blk < 0 || blk >= num_blocks) { ok = 0; break; }
                const uint8_t* rec = pool + (((int64_t)blk * H + h) * 2 + 0) * stride;
                oaken_ref_dequantize_slot(rec, 0, P, d, t % P, thr + (h * 2 + 0) * 4, kv, NULL);
                for (int gq = 0; gq < G; ++gq) {
                    double dot = 0.0;
                    for (int j = 0; j < d; ++j) dot += qd[gq * d + j] * kv[j];
                    sc[(int64_t)gq * Ls + t] = dot * (double)scale;
                }
            }
            if (ok) {
                for (int gq = 0; gq < G; ++gq) {
                    double m = -INFINITY;
                    for (int t = t0; t < Ls; ++t) if (sc[(int64_t)gq * Ls + t] > m) m = sc[(int64_t)gq * Ls + t];
                    double l = 0.0;
                    for (int t = t0; t < Ls; ++t) {
                        double p = exp(sc[(int64_t)gq * Ls + t] - m);
                        sc[(int64_t)gq * Ls + t] = p;
                        l += p;
                    }
                    for (int t = t0; t < Ls; ++t) sc[(int64_t)gq * Ls + t] /= l;
                }
                for (int t = t0; t < Ls; ++t) {
                    int blk = block_table[(int64_t)s * max_blocks + t / P];
                    const uint8_t* rec = pool + (((int64_t)blk * H + h) * 2 + 1) * stride;
                    oaken_ref_dequantize_slot(rec, 1, P, d, t % P, thr + (h * 2 + 1) * 4, kv, NULL);
                    for (int gq = 0; gq < G; ++gq)
                        for (int j = 0; j < d; ++j) acc[gq * d + j] += sc[(int64_t)gq * Ls + t] * kv[j];
                }
                for (int gq = 0; gq < G; ++gq)
                    for (int j = 0; j < d; ++j)
                        out[((int64_t)s * Hq + h * G + gq) * d + j] = (float)acc[gq * d + j];
            } else {
#pragma omp atomic write
                bad = 1;
            }
            free(kv); free(sc); free(acc); free(qd);
        }
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Offline threshold profiling (Sec. 4.3 and Sec. 6.1): per calibration run  */
/* the group boundaries are order statistics of that run's values; the four  */
/* thresholds are the averages over runs.  Outer share r_o is split evenly   */
/* between the two tails; inner share r_i is the r_i fraction of values with */
/* the smallest magnitude, bounded symmetrically by +-t.                     */
/* ------------------------------------------------------------------------ */

static int cmp_float(const void* pa, const void* pb)
{
    float a = *(const float*)pa, b = *(const float*)pb;
    return (a > b) - (a < b);
}

int oaken_ref_calibrate(const uint16_t* k_calib, const uint16_t* v_calib, int R, int T, int H,
                        int d, float r_o, float r_i, float* thr_out)
{
    const int64_t n = (int64_t)T * d;
    if (R < 1 || T < 1 || H < 1 || d < 1) return -1;
    if (!(r_o >= 0.0f && r_o < 1.0f && r_i >= 0.0f && r_i <= 1.0f && r_o + r_i <= 1.0f)) return -1;
    const int64_t k_o = (int64_t)nearbyint((double)n * (double)r_o / 2.0);
    const int64_t k_i = (int64_t)nearbyint((double)n * (double)r_i);
    if (2 * k_o > n - 1 || k_i > n) return -1;
    float* v = (float*)malloc(sizeof(float) * n);
    float* m = (float*)malloc(sizeof(float) * n);
    for (int h = 0; h < H; ++h)
        for (int which = 0; which < 2; ++which) {
            const uint16_t* src = which ? v_calib : k_calib;
            double s_lo = 0.0, s_hi = 0.0, s_t = 0.0;
            for (int r = 0; r < R; ++r) {
                int64_t k = 0;
                for (int t = 0; t < T; ++t)
                    for (int j = 0; j < d; ++j) {
                        float x = oaken_ref_half_to_float(src[(((int64_t)r * T + t) * H + h) * d + j]);
                        v[k] = x;
                        m[k] = fabsf(x);
                        ++k;
                    }
                qsort(v, (size_t)n, sizeof(float), cmp_float);
                qsort(m, (size_t)n, sizeof(float), cmp_float);
                s_lo += v[k_o];
                s_hi += v[n - 1 - k_o];
                s_t += k_i ? m[k_i - 1] : 0.0f;
            }
            float lo_o = (float)(s_lo / (double)R);
            float hi_o = (float)(s_hi / (double)R);
            float t = (float)(s_t / (double)R);
            float lo_i = -t, hi_i = t;
            /* keep lo_o <= lo_i <= hi_i <= hi_o so that Eq. 1's sets partition the line */
            lo_i = fminf(fmaxf(lo_i, lo_o), hi_o);
            hi_i = fmaxf(fminf(hi_i, hi_o), lo_i);
            float out4[4] = {lo_o, lo_i, hi_i, hi_o};
            for (int k = 0; k < 4; ++k)
                thr_out[(h * 2 + which) * 4 + k] = (out4[k] == 0.0f) ? 0.0f : out4[k];
        }
    free(v);
    free(m);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Group-count variants (Sec. 6.2, the number-of-groups study).  The paper    */
/* compares its three groups with two groups (a COO entry of 6 index bits,   */
/* the sign and one pad bit), four or five groups (two group bits: 9-bit COO */
/* entries, padded) and 4-bit outliers (the sign moves into the nibble so    */
/* that the COO entry keeps 8 bits).  The group layout of the four- and      */
/* five-group variants is not given; the reading used here splits the outer */
/* share (and, for five groups, the inner share) into two equal levels, the  */
/* total outlier share staying at 10 %.                                      */
/*                                                                           */
/* thr8 = lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa, hi_ob: outer      */
/* boundaries a (inner) and b (outermost), inner boundaries a (the middle's  */
/* edge) and b (innermost).  Groups, numbered from the inside out: the       */
/* innermost (not shifted), inner a (shifted by ib), middle (shifted by ia,  */
/* or not shifted without inner groups), outer a (shifted by oa), outer b    */
/* (shifted by ob).  A value on a boundary belongs to the inner side, as in  */
/* Eq. 1.  Middle magnitudes have 3 bits; outliers 4 bits, or 3 bits with     */
/* 4-bit outliers.  Codes are offset binary with the side on top, as in the  */
/* three-group quantizer.                                                    */
/*                                                                           */
/* Per vector: nibbles (d/2 bytes, element j in byte j/2, even j low), COO   */
/* entries in chunk then index order (1 or 2 bytes each, little endian),     */
/* per-64-chunk counts, and meta = (Min, Delta) fp16 per group.             */
/* COO entry = side << (6 + gb) | outlier group rank << 6 | index, gb = 1    */
/* for up to two outlier groups and 2 otherwise; without the side bit for    */
/* 4-bit outliers.                                                           */
/* ------------------------------------------------------------------------ */

enum { REF_V3 = 0, REF_V2 = 1, REF_V4 = 2, REF_V5 = 3, REF_V4_O4 = 4, REF_V5_O4 = 5 };

/* out: n_out, n_in, outlier magnitude bits, COO bits, COO bytes, groups. */
int oaken_ref_variant_info(int variant, int out[6])
{
    static const int tab[6][3] = {{1, 1, 4}, {1, 0, 4}, {2, 1, 4}, {2, 2, 4}, {2, 1, 3}, {2, 2, 3}};
    if (variant < 0 || variant > 5) return -1;
    const int n_out = tab[variant][0], n_in = tab[variant][1], ob = tab[variant][2];
    const int n_outlier_groups = n_out + n_in;
    const int gb = n_outlier_groups <= 2 ? 1 : 2;
    const int coo_bits = 6 + gb + (ob == 4 ? 1 : 0);
    out[0] = n_out;
    out[1] = n_in;
    out[2] = ob;
    out[3] = coo_bits;
    out[4] = coo_bits <= 8 ? 1 : 2;
    out[5] = n_in + 1 + n_out;
    return 0;
}

int oaken_ref_variant_quantize_vector(int variant, const uint16_t* x, int d, const float thr8[8],
                                      uint8_t* nib, uint8_t* coo, uint8_t* counts, uint16_t* meta,
                                      int* n_coo)
{
    int info[6];
    if (oaken_ref_variant_info(variant, info) || d < 64 || d % 64) return -1;
    const int n_out = info[0], n_in = info[1], ob = info[2], coo_bits = info[3], cb = info[4], ng = info[5];
    const int gb = coo_bits - 6 - (ob == 4 ? 1 : 0);
    const int mid = n_in;
    const float lo_ob = thr8[0], lo_oa = thr8[1], lo_ia = thr8[2], lo_ib = thr8[3];
    const float hi_ib = thr8[4], hi_ia = thr8[5], hi_oa = thr8[6], hi_ob = thr8[7];
    float* a = (float*)malloc(sizeof(float) * d);
    uint8_t* side = (uint8_t*)malloc(d);
    uint8_t* grp = (uint8_t*)malloc(d);
    uint8_t* code = (uint8_t*)malloc(d);

    for (int j = 0; j < d; ++j) {
        const float xf = oaken_ref_half_to_float(x[j]);
        float t;
        int g, shifted = 1;
        if (n_out == 2 && (xf < lo_ob || xf > hi_ob)) {
            g = mid + 2; side[j] = xf > hi_ob; t = side[j] ? hi_ob : lo_ob;
        } else if (xf < lo_oa || xf > hi_oa) {
            g = mid + 1; side[j] = xf > hi_oa; t = side[j] ? hi_oa : lo_oa;
        } else if (n_in == 0) {
            g = mid; shifted = 0; t = 0.0f;
        } else if (xf < lo_ia || xf > hi_ia) {
            g = mid; side[j] = xf > hi_ia; t = side[j] ? hi_ia : lo_ia;
        } else if (n_in == 2 && (xf < lo_ib || xf > hi_ib)) {
            g = 1; side[j] = xf > hi_ib; t = side[j] ? hi_ib : lo_ib;
        } else {
            g = 0; shifted = 0; t = 0.0f;
        }
        if (!shifted) {
            side[j] = xf >= 0.0f;
            a[j] = fabsf(xf);
        } else {
            a[j] = fabsf(xf - t);
        }
        grp[j] = (uint8_t)g;
    }

    for (int g = 0; g < ng; ++g) {
        float mn = INFINITY, mx = -INFINITY;
        int any = 0;
        for (int j = 0; j < d; ++j)
            if (grp[j] == g) {
                any = 1;
                if (a[j] < mn) mn = a[j];
                if (a[j] > mx) mx = a[j];
            }
        if (!any) { mn = 0.0f; mx = 0.0f; }
        const int bits = (g == mid) ? 3 : ob;
        const int levels = (1 << bits) - 1;
        const float range = mx - mn;
        const float sigma = (range == 0.0f) ? 0.0f : (float)levels / range;   /* Eq. 2 */
        for (int j = 0; j < d; ++j) {
            if (grp[j] != g) continue;
            const float r = rintf((a[j] - mn) * sigma);                        /* Eq. 3 */
            int c = (int)r;
            if (c < 0) c = 0;
            if (c > levels) c = levels;
            code[j] = (uint8_t)(side[j] ? (levels + 1) + c : levels - c);
        }
        meta[2 * g] = oaken_ref_float_to_half(mn);
        meta[2 * g + 1] = oaken_ref_float_to_half(range / (float)levels);
    }

    memset(nib, 0, (size_t)d / 2);
    for (int j = 0; j < d; ++j)
        nib[j / 2] |= (uint8_t)((code[j] & 15) << (4 * (j & 1)));

    int n = 0;
    for (int c = 0; c < d / 64; ++c) {
        int cnt = 0;
        for (int j = c * 64; j < c * 64 + 64; ++j) {
            if (grp[j] == mid) continue;
            /* rank among the outlier groups, from the inside out */
            const int rank = grp[j] < mid ? grp[j] : grp[j] - 1;
            uint32_t e = ((uint32_t)rank << 6) | (uint32_t)(j & 63);
            if (ob == 4) e |= (uint32_t)(code[j] >> 4) << (6 + gb);
            coo[(size_t)n * cb] = (uint8_t)(e & 0xff);
            if (cb == 2) coo[(size_t)n * cb + 1] = (uint8_t)(e >> 8);
            ++n;
            ++cnt;
        }
        counts[c] = (uint8_t)cnt;
    }
    *n_coo = n;
    free(a);
    free(side);
    free(grp);
    free(code);
    return 0;
}

/* Dequantization of one variant-encoded vector, fp64 (the plain definition:
 * the magnitude is Min + c * Delta, the value is the side's threshold plus or
 * minus it, or +-magnitude for unshifted groups). */
int oaken_ref_variant_dequantize_vector(int variant, const uint8_t* nib, const uint8_t* coo,
                                        const uint8_t* counts, const uint16_t* meta, int d,
                                        const float thr8[8], double* out)
{
    int info[6];
    if (oaken_ref_variant_info(variant, info) || d < 64 || d % 64) return -1;
    const int n_out = info[0], n_in = info[1], ob = info[2], coo_bits = info[3], cb = info[4], ng = info[5];
    const int gb = coo_bits - 6 - (ob == 4 ? 1 : 0);
    const int mid = n_in;
    int* u = (int*)malloc(sizeof(int) * d);
    uint8_t* grp = (uint8_t*)malloc(d);
    for (int j = 0; j < d; ++j) {
        u[j] = (nib[j / 2] >> (4 * (j & 1))) & 15;
        grp[j] = (uint8_t)mid;
    }
    int e = 0;
    for (int c = 0; c < d / 64; ++c)
        for (int k = 0; k < counts[c]; ++k, ++e) {
            uint32_t v = coo[(size_t)e * cb];
            if (cb == 2) v |= (uint32_t)coo[(size_t)e * cb + 1] << 8;
            const int j = c * 64 + (int)(v & 63);
            const int rank = (int)((v >> 6) & ((1u << gb) - 1));
            grp[j] = (uint8_t)(rank < mid ? rank : rank + 1);
            if (ob == 4) u[j] |= (int)((v >> (6 + gb)) & 1) << 4;
        }
    const double th[8] = {thr8[0], thr8[1], thr8[2], thr8[3], thr8[4], thr8[5], thr8[6], thr8[7]};
    for (int j = 0; j < d; ++j) {
        const int g = grp[j];
        if (g >= ng) { free(u); free(grp); return -1; }
        const int bits = (g == mid) ? 3 : ob;
        const int half = 1 << bits;
        const int hi = u[j] >> bits;
        const int c = hi ? u[j] - half : half - 1 - u[j];
        const double mag = (double)oaken_ref_half_to_float(meta[2 * g]) +
                           (double)c * (double)oaken_ref_half_to_float(meta[2 * g + 1]);
        double lo_t, hi_t;
        if (g == mid + 2)                { lo_t = th[0]; hi_t = th[7]; }
        else if (g == mid + 1)           { lo_t = th[1]; hi_t = th[6]; }
        else if (g == mid && n_in > 0)   { lo_t = th[2]; hi_t = th[5]; }
        else if (g == 1 && n_in == 2)    { lo_t = th[3]; hi_t = th[4]; }
        else                             { lo_t = 0.0; hi_t = 0.0; }
        out[j] = hi ? hi_t + mag : lo_t - mag;
    }
    (void)n_out;
    free(u);
    free(grp);
    return 0;
}

/* Batch over [n][H] vectors; thr8 per head ([H][8]), outputs laid out per vector:
 * nib [n][H][d/2], coo [n][H][d * coo_bytes], counts [n][H][d/64], meta [n][H][2 * groups],
 * n_coo [n][H]. */
int oaken_ref_variant_quantize(int variant, const uint16_t* x, int n, int H, int d, const float* thr8,
                               uint8_t* nib, uint8_t* coo, uint8_t* counts, uint16_t* meta, int32_t* n_coo)
{
    int info[6];
    if (oaken_ref_variant_info(variant, info) || d < 64 || d % 64) return -1;
    const int cb = info[4], ng = info[5];
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (int64_t v = 0; v < (int64_t)n * H; ++v) {
        const int h = (int)(v % H);
        int nc = 0;
        bad |= oaken_ref_variant_quantize_vector(variant, x + v * d, d, thr8 + 8 * h, nib + v * (d / 2),
                                                 coo + v * d * cb, counts + v * (d / 64), meta + v * 2 * ng, &nc);
        n_coo[v] = nc;
    }
    return bad ? -1 : 0;
}

int oaken_ref_variant_dequantize(int variant, const uint8_t* nib, const uint8_t* coo, const uint8_t* counts,
                                 const uint16_t* meta, int n, int H, int d, const float* thr8, double* out)
{
    int info[6];
    if (oaken_ref_variant_info(variant, info) || d < 64 || d % 64) return -1;
    const int cb = info[4], ng = info[5];
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (int64_t v = 0; v < (int64_t)n * H; ++v) {
        const int h = (int)(v % H);
        bad |= oaken_ref_variant_dequantize_vector(variant, nib + v * (d / 2), coo + v * d * cb, counts + v * (d / 64),
                                                   meta + v * 2 * ng, d, thr8 + 8 * h, out + v * d);
    }
    return bad ? -1 : 0;
}

/* Thread count of the parallel loops (timing of the CPU baseline at 1 and at all
   cores); n <= 0 leaves it unchanged. */
void oaken_ref_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int oaken_ref_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
