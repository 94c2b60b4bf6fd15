/*
 * tco.c -- CPU oracle for the boundary compressors of
 *   M. Rudakov, A. Beznosikov, Y. Kholodov, A. Gasnikov,
 *   "Activations and Gradients Compression for Model-Parallel Training" (2024).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain reference that the
 * GPU library is checked against.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  It shares no code, header,
 * table or helper with the GPU library, and it includes nothing from it.
 *
 * Every routine below writes out a definition from the paper directly:
 *   - TopK (Sec. 2.3): keep the K% entries of largest absolute value and zero
 *     the rest; the indices travel with the values (Sec. 4.1 notes that
 *     sparsification has to send the indices along with the data).
 *   - uniform b-bit quantization with min-max scaling (Sec. 2.2): map the
 *     vector to [0,1] with its min and max, quantize to 2^b levels, and
 *     decompress back to the original scale.
 *   - error feedback (Sec. 2.4): e = X - C(X); the next round sends C(X + e),
 *     with one global buffer per compression operator.
 *   - EF-mixed (Sec. 2.4): half of the TopK budget on the input, half on the
 *     error buffer; both lists are sent and added by the receiver.
 *   - AQ-SGD (Sec. 2.5): a buffer per training example; the change of the
 *     activation against that buffer is compressed and sent, and both sides
 *     add the sent message to their copy of the buffer.
 *
 * Readings where the paper is silent (tie order, rounding mode, bit order of
 * the packed codes, -0, the k for a percentage) are stated at each routine.
 *
 * Build: gcc -std=c11 -O2 -ffp-contract=off -fno-fast-math -fopenmp -fPIC
 * (no FMA contraction, no flush-to-zero: IEEE single precision throughout).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* dtype codes for raw element buffers handed to the oracle */
enum { TCO_F32 = 0, TCO_BF16 = 1, TCO_F16 = 2 };

/* ------------------------------------------------------------------------ */
/* Floating-point formats (IEEE 754 binary32, binary16; bfloat16 is binary32  */
/* with the low 16 fraction bits removed).  The conversions are written from  */
/* the definition of round-to-nearest, ties-to-even: every finite binary32   */
/* value and every midpoint between neighbouring narrow values is exact in   */
/* binary64, so the rounding decision below is taken on exact numbers.       */
/* ------------------------------------------------------------------------ */

static float f32_from_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t bits_from_f32(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* round a nonnegative exact multiple count n (n = a / q, q a power of two) to
 * the nearest integer, ties to even */
static double round_half_even(double n) {
    double fl = floor(n);
    double fr = n - fl;              /* exact: n has few significant bits */
    if (fr > 0.5) return fl + 1.0;
    if (fr < 0.5) return fl;
    return (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
}

float tco_f16_to_f32(uint16_t h) {
    uint32_t sign = (h >> 15) & 1u, ex = (h >> 10) & 0x1Fu, man = h & 0x3FFu;
    double v;
    if (ex == 0x1F) {
        if (man) return f32_from_bits(0x7FC00000u | (sign << 31));
        v = INFINITY;
    } else if (ex == 0) {
        v = ldexp((double)man, -24);            /* subnormal: man * 2^-24 */
    } else {
        v = ldexp((double)(1024u + man), (int)ex - 25);
    }
    return (float)(sign ? -v : v);
}

uint16_t tco_f32_to_f16(float f) {
    uint32_t u = bits_from_f32(f);
    uint16_t sign = (uint16_t)((u >> 31) << 15);
    if (isnan(f)) return (uint16_t)(sign | 0x7E00u);
    double a = fabs((double)f);
    /* 65520 is the midpoint between 65504 (largest finite, odd fraction) and
     * 2^16; the tie goes to the even neighbour 2^16, which overflows. */
    if (a >= 65520.0) return (uint16_t)(sign | 0x7C00u);
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);                      /* a = m * 2^e, m in [0.5,1) */
    int unb = e - 1;                   /* a in [2^unb, 2^(unb+1)) */
    if (unb < -14) unb = -14;          /* subnormal range shares the 2^-24 quantum */
    double q = ldexp(1.0, unb - 10);
    double r = round_half_even(a / q) * q;   /* the nearest representable value */
    if (r == 0.0) return sign;
    if (r < ldexp(1.0, -14)) {               /* subnormal result */
        return (uint16_t)(sign | (uint16_t)(r / ldexp(1.0, -24)));
    }
    frexp(r, &e);
    int ex = e - 1;                           /* may have carried into the next binade */
    double man = r / ldexp(1.0, ex) * 1024.0 - 1024.0;
    return (uint16_t)(sign | (uint16_t)((ex + 15) << 10) | (uint16_t)man);
}

float tco_bf16_to_f32(uint16_t h) { return f32_from_bits((uint32_t)h << 16); }

uint16_t tco_f32_to_bf16(float f) {
    uint32_t u = bits_from_f32(f);
    uint16_t sign = (uint16_t)((u >> 31) << 15);
    if (isnan(f)) return (uint16_t)(sign | 0x7FC0u);
    double a = fabs((double)f);
    /* largest finite bfloat16 is (2 - 2^-7) * 2^127 (odd fraction); the midpoint
     * to 2^128 is (2 - 2^-8) * 2^127 and rounds to the even side, i.e. overflows */
    if (a >= ldexp(2.0 - ldexp(1.0, -8), 127)) return (uint16_t)(sign | 0x7F80u);
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);
    int unb = e - 1;
    if (unb < -126) unb = -126;          /* subnormal quantum 2^-133 */
    double q = ldexp(1.0, unb - 7);
    double r = round_half_even(a / q) * q;
    if (r == 0.0) return sign;
    /* r is exactly representable in binary32 and, by construction, has at most
     * 8 significant bits; its binary32 pattern therefore ends in 16 zero bits */
    uint32_t rb = bits_from_f32((float)r);
    return (uint16_t)(sign | (uint16_t)(rb >> 16));
}

/* element i of a raw buffer of the given dtype, as binary32 (exact) */
static float load_f32(const void* p, int dt, uint64_t i) {
    if (dt == TCO_F32) return ((const float*)p)[i];
    if (dt == TCO_BF16) return tco_bf16_to_f32(((const uint16_t*)p)[i]);
    return tco_f16_to_f32(((const uint16_t*)p)[i]);
}

/* store binary32 v rounded to nearest-even into element i of the given dtype */
static void store_rne(void* p, int dt, uint64_t i, float v) {
    if (dt == TCO_F32) ((float*)p)[i] = v;
    else if (dt == TCO_BF16) ((uint16_t*)p)[i] = tco_f32_to_bf16(v);
    else ((uint16_t*)p)[i] = tco_f32_to_f16(v);
}

/* the value a receiver holds after the value v went through dtype dt */
static float through(int dt, float v) {
    if (dt == TCO_F32) return v;
    if (dt == TCO_BF16) return tco_bf16_to_f32(tco_f32_to_bf16(v));
    return tco_f16_to_f32(tco_f32_to_f16(v));
}

/* ------------------------------------------------------------------------ */
/* TopK (Sec. 2.3)                                                            */
/* ------------------------------------------------------------------------ */

/* k for "K percent" of L entries given as the fraction num/den: the smallest
 * integer not below L*num/den, computed in integers (a binary fraction such
 * as 0.3 is not exact, and its ceiling can come out one too high). */
uint64_t tco_topk_count(uint64_t L, uint32_t num, uint32_t den) {
    if (den == 0) return 0;
    unsigned __int128 p = (unsigned __int128)L * num + (den - 1);
    return (uint64_t)(p / den);
}

typedef struct { float mag; uint32_t idx; } mag_idx;

/* order: larger |v| first; equal |v| (including +0 against -0): lower index
 * first.  The paper fixes no tie order; lowest index first is our reading. */
static int by_mag_desc_idx_asc(const void* pa, const void* pb) {
    const mag_idx* a = (const mag_idx*)pa;
    const mag_idx* b = (const mag_idx*)pb;
    if (a->mag > b->mag) return -1;
    if (a->mag < b->mag) return 1;
    return (a->idx < b->idx) ? -1 : (a->idx > b->idx);
}

static int u32_asc(const void* pa, const void* pb) {
    uint32_t a = *(const uint32_t*)pa, b = *(const uint32_t*)pb;
    return (a > b) - (a < b);
}

/* Indices (ascending) of the k entries of v[0..L) with the largest absolute
 * values.  Returns 0 on success, -1 on bad arguments or allocation failure. */
int tco_topk_indices(const float* v, uint64_t L, uint64_t k, uint32_t* idx) {
    if (k > L || L > 0xFFFFFFFFull) return -1;
    if (k == 0) return 0;
    mag_idx* t = (mag_idx*)malloc(sizeof(mag_idx) * (size_t)L);
    if (!t) return -1;
    for (uint64_t i = 0; i < L; ++i) { t[i].mag = fabsf(v[i]); t[i].idx = (uint32_t)i; }
    qsort(t, (size_t)L, sizeof(mag_idx), by_mag_desc_idx_asc);
    for (uint64_t j = 0; j < k; ++j) idx[j] = t[j].idx;
    free(t);
    qsort(idx, (size_t)k, sizeof(uint32_t), u32_asc);
    return 0;
}

/* TopK compression of n_seg independent segments of length L (each a sample,
 * a token row, or the whole tensor).  x has dtype dt; kept values are sent in
 * dtype wire (rounded to nearest-even).  idx/val are [n_seg][k]. */
int tco_topk_compress(const void* x, int dt, uint64_t n_seg, uint64_t L, uint64_t k,
                      int wire, uint32_t* idx, void* val, int threads) {
    int bad = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 1) reduction(|: bad)
#endif
    for (long long s = 0; s < (long long)n_seg; ++s) {
        float* v = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
        if (!v) { bad |= 1; continue; }
        for (uint64_t i = 0; i < L; ++i) v[i] = load_f32(x, dt, (uint64_t)s * L + i);
        uint32_t* id = idx + (uint64_t)s * k;
        if (tco_topk_indices(v, L, k, id) != 0) bad |= 1;
        else for (uint64_t j = 0; j < k; ++j) store_rne(val, wire, (uint64_t)s * k + j, v[id[j]]);
        free(v);
    }
    return bad ? -1 : 0;
}

/* Receiver side of TopK: a dense tensor that is +0 everywhere except at the
 * sent indices, which hold the sent values converted to out_dt. */
int tco_topk_decompress(const uint32_t* idx, const void* val, int wire, uint64_t n_seg,
                        uint64_t L, uint64_t k, void* y, int out_dt) {
    for (uint64_t s = 0; s < n_seg; ++s) {
        for (uint64_t i = 0; i < L; ++i) store_rne(y, out_dt, s * L + i, 0.0f);
        for (uint64_t j = 0; j < k; ++j) {
            uint32_t i = idx[s * k + j];
            if (i >= L) return -1;
            store_rne(y, out_dt, s * L + i, load_f32(val, wire, s * k + j));
        }
    }
    return 0;
}

/* TopK at given indices (Sec. 3.2, the GPT-2 fine-tuning runs: gradients are
 * compressed at the indices that the TopK of the activations kept, rather
 * than by a selection of their own; compressing them separately made those
 * runs diverge).  The message is x at those indices, in index order, in the
 * wire dtype; the receiver is tco_topk_decompress with the same indices.
 * With e (non-NULL) it is the Sec. 2.4 error-feedback sender around this
 * compressor: X = x + e is compressed and e becomes X minus what the
 * receiver holds (the wire value of X at the indices, +0 elsewhere).  An
 * index outside the segment is an error. */
int tco_topk_gather(const void* x, int dt, float* e, uint64_t n_seg, uint64_t L, uint64_t k,
                    const uint32_t* idx, int wire, void* val) {
    float* X = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
    float* r = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
    if (!X || !r) { free(X); free(r); return -1; }
    int bad = 0;
    for (uint64_t s = 0; s < n_seg && !bad; ++s) {
        const uint64_t base = s * L;
        for (uint64_t i = 0; i < L; ++i) {
            X[i] = load_f32(x, dt, base + i);
            if (e) X[i] = X[i] + e[base + i];
            r[i] = 0.0f;
        }
        for (uint64_t j = 0; j < k; ++j) {
            const uint32_t i = idx[s * k + j];
            if (i >= L) { bad = 1; break; }
            store_rne(val, wire, s * k + j, X[i]);
            r[i] = load_f32(val, wire, s * k + j);
        }
        if (!bad && e)
            for (uint64_t i = 0; i < L; ++i) e[base + i] = X[i] - r[i];
    }
    free(X); free(r);
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Uniform b-bit min-max quantization (Sec. 2.2)                             */
/* ------------------------------------------------------------------------ */

/* bytes taken by one group's codes: whole 32-bit words, zero padded */
uint64_t tco_quant_group_bytes(uint64_t G, uint32_t b) {
    return 4u * ((G * b + 31u) / 32u);
}

static void put_bits(uint8_t* stream, uint64_t bitpos, uint32_t code, uint32_t b) {
    for (uint32_t j = 0; j < b; ++j)
        if ((code >> j) & 1u) stream[(bitpos + j) >> 3] |= (uint8_t)(1u << ((bitpos + j) & 7u));
}

static uint32_t get_bits(const uint8_t* stream, uint64_t bitpos, uint32_t b) {
    uint32_t c = 0;
    for (uint32_t j = 0; j < b; ++j)
        c |= (uint32_t)((stream[(bitpos + j) >> 3] >> ((bitpos + j) & 7u)) & 1u) << j;
    return c;
}

/* Quantize one group v[0..G) to b bits (1 <= b <= 8), or pass it through raw
 * when b == 32 (the paper's "no compression" rows).
 *   lo, hi  = min and max of the group (a -0 is read as +0);
 *   u       = (v - lo) / (hi - lo)            -- the map onto [0,1];
 *   code    = round-half-even(u * (2^b - 1))   -- 2^b levels;
 *   meta    = (lo, scale) with scale = (hi - lo) / (2^b - 1);
 * a group whose entries are all equal gets codes 0 and scale 0.  Codes are
 * written LSB-first into a little-endian bit stream of tco_quant_group_bytes. */
int tco_quant_group(const float* v, uint64_t G, uint32_t b, uint8_t* codes, float* meta) {
    if (b == 32) {
        memcpy(codes, v, (size_t)G * 4u);
        meta[0] = 0.0f; meta[1] = 0.0f;
        return 0;
    }
    if (b < 1 || b > 8) return -1;
    memset(codes, 0, (size_t)tco_quant_group_bytes(G, b));
    if (G == 0) { meta[0] = 0.0f; meta[1] = 0.0f; return 0; }
    float lo = v[0], hi = v[0];
    for (uint64_t i = 1; i < G; ++i) { if (v[i] < lo) lo = v[i]; if (v[i] > hi) hi = v[i]; }
    lo = lo + 0.0f;      /* -0 + +0 = +0 under round-to-nearest */
    hi = hi + 0.0f;
    const uint32_t levels = (1u << b) - 1u;
    meta[0] = lo;
    if (hi == lo) { meta[1] = 0.0f; return 0; }
    const float range = hi - lo;
    meta[1] = range / (float)levels;
    for (uint64_t i = 0; i < G; ++i) {
        float u = (v[i] - lo) / range;
        float t = u * (float)levels;
        uint32_t c = (uint32_t)rintf(t);
        if (c > levels) c = levels;
        put_bits(codes, i * b, c, b);
    }
    return 0;
}

/* Decompression: xhat = lo + code * scale (a product, then a sum, each rounded
 * to binary32), stored to out_dt. */
int tco_dequant_group(const uint8_t* codes, const float* meta, uint64_t G, uint32_t b,
                      void* y, int out_dt, uint64_t y_off) {
    if (b == 32) {
        const float* raw = (const float*)codes;
        for (uint64_t i = 0; i < G; ++i) store_rne(y, out_dt, y_off + i, raw[i]);
        return 0;
    }
    if (b < 1 || b > 8) return -1;
    for (uint64_t i = 0; i < G; ++i) {
        float prod = (float)get_bits(codes, i * b, b) * meta[1];
        float xh = meta[0] + prod;
        store_rne(y, out_dt, y_off + i, xh);
    }
    return 0;
}

/* n_grp groups of G entries of x (dtype dt), codes [n_grp][group_bytes] and
 * meta [n_grp][2] */
int tco_quant_pack(const void* x, int dt, uint64_t n_grp, uint64_t G, uint32_t b,
                   uint8_t* codes, float* meta, int threads) {
    const uint64_t gb = (b == 32) ? G * 4u : tco_quant_group_bytes(G, b);
    int bad = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 1) reduction(|: bad)
#endif
    for (long long g = 0; g < (long long)n_grp; ++g) {
        float* v = (float*)malloc(sizeof(float) * (size_t)(G ? G : 1));
        if (!v) { bad |= 1; continue; }
        for (uint64_t i = 0; i < G; ++i) v[i] = load_f32(x, dt, (uint64_t)g * G + i);
        if (tco_quant_group(v, G, b, codes + (uint64_t)g * gb, meta + 2u * (uint64_t)g) != 0) bad |= 1;
        free(v);
    }
    return bad ? -1 : 0;
}

int tco_quant_unpack(const uint8_t* codes, const float* meta, uint64_t n_grp, uint64_t G,
                     uint32_t b, void* y, int out_dt) {
    const uint64_t gb = (b == 32) ? G * 4u : tco_quant_group_bytes(G, b);
    for (uint64_t g = 0; g < n_grp; ++g)
        if (tco_dequant_group(codes + g * gb, meta + 2u * g, G, b, y, out_dt, g * G) != 0) return -1;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Error feedback (Sec. 2.4)                                                  */
/*   X = x + e;  send C(X);  e <- X - D(C(X))                                 */
/* where D(C(X)) is exactly what the receiver's dense tensor holds, read back */
/* as binary32.  One buffer per compression operator, carried to the next     */
/* batch of the same shape; it starts at zero.                                */
/* ------------------------------------------------------------------------ */

/* EF around TopK: x (dt) and e (binary32) are [n_seg][L]; payload idx/val in
 * dtype wire.  The receiver's value at a kept index is wire(X), else +0. */
int tco_ef_topk(const void* x, int dt, float* e, uint64_t n_seg, uint64_t L, uint64_t k,
                int wire, uint32_t* idx, void* val, int threads) {
    int bad = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 1) reduction(|: bad)
#endif
    for (long long s = 0; s < (long long)n_seg; ++s) {
        const uint64_t base = (uint64_t)s * L;
        float* X = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
        float* r = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
        if (!X || !r) { free(X); free(r); bad |= 1; continue; }
        for (uint64_t i = 0; i < L; ++i) { X[i] = load_f32(x, dt, base + i) + e[base + i]; r[i] = 0.0f; }
        uint32_t* id = idx + (uint64_t)s * k;
        if (tco_topk_indices(X, L, k, id) != 0) { bad |= 1; }
        else {
            for (uint64_t j = 0; j < k; ++j) {
                store_rne(val, wire, (uint64_t)s * k + j, X[id[j]]);
                r[id[j]] = load_f32(val, wire, (uint64_t)s * k + j);
            }
            for (uint64_t i = 0; i < L; ++i) e[base + i] = X[i] - r[i];
        }
        free(X); free(r);
    }
    return bad ? -1 : 0;
}

/* EF around min-max quantization: groups of G entries; the receiver holds
 * out_dt(lo + code*scale). */
int tco_ef_quant(const void* x, int dt, float* e, uint64_t n_grp, uint64_t G, uint32_t b,
                 int out_dt, uint8_t* codes, float* meta, int threads) {
    const uint64_t gb = (b == 32) ? G * 4u : tco_quant_group_bytes(G, b);
    int bad = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 1) reduction(|: bad)
#endif
    for (long long g = 0; g < (long long)n_grp; ++g) {
        const uint64_t base = (uint64_t)g * G;
        float* X = (float*)malloc(sizeof(float) * (size_t)(G ? G : 1));
        void* y = malloc(4u * (size_t)(G ? G : 1));
        if (!X || !y) { free(X); free(y); bad |= 1; continue; }
        for (uint64_t i = 0; i < G; ++i) X[i] = load_f32(x, dt, base + i) + e[base + i];
        uint8_t* cg = codes + (uint64_t)g * gb;
        float* mg = meta + 2u * (uint64_t)g;
        if (tco_quant_group(X, G, b, cg, mg) != 0 || tco_dequant_group(cg, mg, G, b, y, out_dt, 0) != 0) {
            bad |= 1;
        } else {
            for (uint64_t i = 0; i < G; ++i) e[base + i] = X[i] - load_f32(y, out_dt, i);
        }
        free(X); free(y);
    }
    return bad ? -1 : 0;
}

/* EF around TopK whose kept list is then min-max quantized as one group per
 * segment (TopK followed by the quantizer of Sec. 2.2 on the kept values).
 * codes [n_seg][group_bytes(k,b)], meta [n_seg][2].  The receiver holds
 * out_dt(lo + code_j*scale) at idx_j and +0 elsewhere. */
int tco_ef_topk_quant(const void* x, int dt, float* e, uint64_t n_seg, uint64_t L, uint64_t k,
                      uint32_t b, int out_dt, uint32_t* idx, uint8_t* codes, float* meta,
                      int threads) {
    const uint64_t gb = (b == 32) ? k * 4u : tco_quant_group_bytes(k, b);
    int bad = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 1) reduction(|: bad)
#endif
    for (long long s = 0; s < (long long)n_seg; ++s) {
        const uint64_t base = (uint64_t)s * L;
        float* X = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
        float* kept = (float*)malloc(sizeof(float) * (size_t)(k ? k : 1));
        void* yk = malloc(4u * (size_t)(k ? k : 1));
        if (!X || !kept || !yk) { free(X); free(kept); free(yk); bad |= 1; continue; }
        for (uint64_t i = 0; i < L; ++i) X[i] = load_f32(x, dt, base + i) + e[base + i];
        uint32_t* id = idx + (uint64_t)s * k;
        uint8_t* cg = codes + (uint64_t)s * gb;
        float* mg = meta + 2u * (uint64_t)s;
        if (tco_topk_indices(X, L, k, id) != 0) { bad |= 1; }
        else {
            for (uint64_t j = 0; j < k; ++j) kept[j] = X[id[j]];
            if (tco_quant_group(kept, k, b, cg, mg) != 0 || tco_dequant_group(cg, mg, k, b, yk, out_dt, 0) != 0) {
                bad |= 1;
            } else {
                /* e <- X - r, with r = +0 off the kept set */
                for (uint64_t i = 0; i < L; ++i) e[base + i] = X[i] - 0.0f;
                for (uint64_t j = 0; j < k; ++j) e[base + id[j]] = X[id[j]] - load_f32(yk, out_dt, j);
            }
        }
        free(X); free(kept); free(yk);
    }
    return bad ? -1 : 0;
}

/* receiver of tco_ef_topk_quant: dense y [n_seg][L] in out_dt */
int tco_topk_quant_decompress(const uint32_t* idx, const uint8_t* codes, const float* meta,
                              uint64_t n_seg, uint64_t L, uint64_t k, uint32_t b,
                              void* y, int out_dt) {
    const uint64_t gb = (b == 32) ? k * 4u : tco_quant_group_bytes(k, b);
    float* yk = (float*)malloc(sizeof(float) * (size_t)(k ? k : 1));
    if (!yk) return -1;
    for (uint64_t s = 0; s < n_seg; ++s) {
        if (tco_dequant_group(codes + s * gb, meta + 2u * s, k, b, yk, TCO_F32, 0) != 0) { free(yk); return -1; }
        for (uint64_t i = 0; i < L; ++i) store_rne(y, out_dt, s * L + i, 0.0f);
        for (uint64_t j = 0; j < k; ++j) {
            uint32_t i = idx[s * k + j];
            if (i >= L) { free(yk); return -1; }
            store_rne(y, out_dt, s * L + i, yk[j]);
        }
    }
    free(yk);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* AQ-SGD with TopK (Sec. 2.5)                                                */
/*   sender:   d = a - m[id];  (idx, v) = TopK(d) sent in the buffer dtype;   */
/*             m[id][idx] <- m[id][idx] + v                                   */
/*   receiver: m'[id][idx] <- m'[id][idx] + v;  a_hat = m'[id]                */
/* The sender adds the value as sent (after rounding to the buffer dtype), so */
/* that both copies of the buffer stay identical.                             */
/* a is [n_ids][L]; m is [n_samples][L]; both in dtype dt.                   */
/* ------------------------------------------------------------------------ */

int tco_aqsgd_send(const void* a, void* m, int dt, uint64_t n_samples, uint64_t L,
                   const int64_t* ids, uint64_t n_ids, uint64_t k,
                   uint32_t* idx, void* val, int threads) {
    for (uint64_t b = 0; b < n_ids; ++b)
        if (ids[b] < 0 || (uint64_t)ids[b] >= n_samples) return -1;
    int bad = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 1) reduction(|: bad)
#endif
    for (long long b = 0; b < (long long)n_ids; ++b) {
        const uint64_t row = (uint64_t)ids[b] * L;
        float* d = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
        if (!d) { bad |= 1; continue; }
        for (uint64_t i = 0; i < L; ++i)
            d[i] = load_f32(a, dt, (uint64_t)b * L + i) - load_f32(m, dt, row + i);
        uint32_t* id = idx + (uint64_t)b * k;
        if (tco_topk_indices(d, L, k, id) != 0) { bad |= 1; }
        else {
            for (uint64_t j = 0; j < k; ++j) {
                const uint64_t o = (uint64_t)b * k + j;
                store_rne(val, dt, o, d[id[j]]);
                store_rne(m, dt, row + id[j], load_f32(m, dt, row + id[j]) + load_f32(val, dt, o));
            }
        }
        free(d);
    }
    return bad ? -1 : 0;
}

int tco_aqsgd_recv(const uint32_t* idx, const void* val, void* m_r, int dt, uint64_t n_samples,
                   uint64_t L, const int64_t* ids, uint64_t n_ids, uint64_t k, void* a_hat) {
    for (uint64_t b = 0; b < n_ids; ++b) {
        if (ids[b] < 0 || (uint64_t)ids[b] >= n_samples) return -1;
        const uint64_t row = (uint64_t)ids[b] * L;
        for (uint64_t j = 0; j < k; ++j) {
            uint32_t i = idx[b * k + j];
            if (i >= L) return -1;
            store_rne(m_r, dt, row + i, load_f32(m_r, dt, row + i) + load_f32(val, dt, b * k + j));
        }
        for (uint64_t i = 0; i < L; ++i) store_rne(a_hat, dt, b * L + i, load_f32(m_r, dt, row + i));
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* EF-mixed (Sec. 2.4): half of the K% budget goes to the largest entries of */
/* the input, the other half to the largest entries of the error buffer.     */
/* The paper does not spell out the arithmetic; our reading:                 */
/*   k_x = k - floor(k/2) entries of x (the input gets the odd one),        */
/*   k_e = floor(k/2) entries of e, each picked by tco_topk_indices on its   */
/*   own vector (the sets may overlap);                                      */
/*   the message is the two lists, each in x's dtype (dt); the receiver's    */
/*   dense tensor starts at +0, takes the x list's values at its indices and */
/*   then adds the e list's values at its indices (binary32 sum, rounded     */
/*   once to out_dt), so the sent tensor is C_kx(x) + C_ke(e);               */
/*   the buffer becomes everything not sent:                                 */
/*     e'_i = (x_i - [i in S_x] dt(x_i)) + (e_i - [i in S_e] dt(e_i) + c_i)  */
/*   in binary32, which is x + e minus what the receiver holds.  c_i is 0    */
/*   except where both lists hold i: there the receiver's tensor (in the     */
/*   wire dtype dt) holds u_i = x_i + dt(e_i) (binary32 sum) rounded once to */
/*   dt, so the part that rounding drops, c_i = u_i - dt(u_i), stays behind. */
/* x is [n_seg][L] of dtype dt; e (binary32) is updated in place; idx_x /   */
/* val_x are [n_seg][k_x], idx_e / val_e are [n_seg][k_e].                  */
/* ------------------------------------------------------------------------ */
uint64_t tco_efmix_kx(uint64_t k) { return k - k / 2; }
uint64_t tco_efmix_ke(uint64_t k) { return k / 2; }

int tco_efmix_send(const void* x, int dt, float* e, uint64_t n_seg, uint64_t L, uint64_t k,
                   uint32_t* idx_x, void* val_x, uint32_t* idx_e, void* val_e) {
    const uint64_t kx = tco_efmix_kx(k), ke = tco_efmix_ke(k);
    if (k > L) return -1;
    float* xv = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
    float* ev = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
    uint8_t* in_x = (uint8_t*)malloc((size_t)(L ? L : 1));
    uint8_t* in_e = (uint8_t*)malloc((size_t)(L ? L : 1));
    int bad = (!xv || !ev || !in_x || !in_e);
    for (uint64_t s = 0; s < n_seg && !bad; ++s) {
        const uint64_t base = s * L;
        for (uint64_t i = 0; i < L; ++i) {
            xv[i] = load_f32(x, dt, base + i);
            ev[i] = e[base + i];
            in_x[i] = in_e[i] = 0;
        }
        uint32_t* ix = idx_x + s * kx;
        uint32_t* ie = idx_e + s * ke;
        if (tco_topk_indices(xv, L, kx, ix) != 0 || tco_topk_indices(ev, L, ke, ie) != 0) { bad = 1; break; }
        for (uint64_t j = 0; j < kx; ++j) { store_rne(val_x, dt, s * kx + j, xv[ix[j]]); in_x[ix[j]] = 1; }
        for (uint64_t j = 0; j < ke; ++j) { store_rne(val_e, dt, s * ke + j, ev[ie[j]]); in_e[ie[j]] = 1; }
        for (uint64_t i = 0; i < L; ++i) {
            const float rx = xv[i] - (in_x[i] ? through(dt, xv[i]) : 0.0f);
            float re = ev[i] - (in_e[i] ? through(dt, ev[i]) : 0.0f);
            if (in_x[i] && in_e[i]) {
                const float u = through(dt, xv[i]) + through(dt, ev[i]);   /* the receiver's sum */
                re = re + (u - through(dt, u));
            }
            e[base + i] = rx + re;
        }
    }
    free(xv); free(ev); free(in_x); free(in_e);
    return bad ? -1 : 0;
}

int tco_efmix_recv(const uint32_t* idx_x, const void* val_x, const uint32_t* idx_e, const void* val_e,
                   int wire, uint64_t n_seg, uint64_t L, uint64_t k, void* y, int out_dt) {
    const uint64_t kx = tco_efmix_kx(k), ke = tco_efmix_ke(k);
    float* d = (float*)malloc(sizeof(float) * (size_t)(L ? L : 1));
    if (!d) return -1;
    int bad = 0;
    for (uint64_t s = 0; s < n_seg && !bad; ++s) {
        for (uint64_t i = 0; i < L; ++i) d[i] = 0.0f;
        for (uint64_t j = 0; j < kx && !bad; ++j) {
            const uint32_t i = idx_x[s * kx + j];
            if (i >= L) bad = 1;
            else d[i] = load_f32(val_x, wire, s * kx + j);
        }
        for (uint64_t j = 0; j < ke && !bad; ++j) {
            const uint32_t i = idx_e[s * ke + j];
            if (i >= L) bad = 1;
            else d[i] = d[i] + load_f32(val_e, wire, s * ke + j);
        }
        for (uint64_t i = 0; i < L && !bad; ++i) store_rne(y, out_dt, s * L + i, d[i]);
    }
    free(d);
    return bad ? -1 : 0;
}

/* helpers for tests: bulk conversions (exact upcast, RNE downcast) */
void tco_to_f32(const void* x, int dt, uint64_t n, float* out) {
    for (uint64_t i = 0; i < n; ++i) out[i] = load_f32(x, dt, i);
}
void tco_from_f32(const float* x, uint64_t n, int dt, void* out) {
    for (uint64_t i = 0; i < n; ++i) store_rne(out, dt, i, x[i]);
}
float tco_through(int dt, float v) { return through(dt, v); }
