/*
 * bytecomp_oracle.c -- plain, slow CPU oracle for the gradient-compression
 * hot path of ByteComp (Wang, Lin, Zhu, Ng: "ByteComp: Revisiting Gradient
 * Compression in Distributed Training", arXiv 2205.14465).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  The product path (the
 * HIP library under paper_2205_14465_amd/csrc) shares no code, header,
 * table or helper with this file, and never calls it.
 *
 * What the paper fixes and what this file reads into it:
 *   - Sparsification sends a subset of the gradient entries; quantization
 *     maps fp32 gradients to fewer bits, down to one bit; both are combined
 *     with error feedback (paper Sec. 2.3, "Gradient Compression").
 *   - The evaluated operators are Randomk and DGC at a 1% rate and
 *     EFSignSGD, with error feedback on every compression (paper Sec. 5.1,
 *     "Compression algorithms").
 *   - Quantization to 8 bits and to 2 bits (TernGrad) is named beside the
 *     1-bit kind (paper Sec. 2.3) but not evaluated; the stochastic
 *     quantizers at the end of this file are a stated reading of the
 *     cited works.
 *   - In an indivisible scheme every node decompresses the N payloads it
 *     gathered and aggregates them; compressed aggregation is not
 *     associative, so it cannot be an Allreduce (paper Sec. 3.1, Reason #2
 *     and the indivisible-scheme figure; Sec. 4.2.1, Dimension 3).
 *   The paper gives no operator formula, so every detail below (k rule,
 *   tie-break, sign convention, scale, summation order, index generator) is
 *   a stated reading; the design notes list each one.
 *
 * Arithmetic: fp32 where the gradients are fp32, IEEE round-to-nearest-even,
 * compiled with -O2 -ffp-contract=off (no FMA contraction, no fast-math).
 * The mean-|v| scale is accumulated in fp64 in index order.  The sparse
 * aggregate adds the workers' values in worker order in fp32; the sign
 * aggregate (and the 2-bit one) is the exact sum of the decoded values
 * rounded once (a 320-bit fixed-point sum), with an order-free rule for
 * non-finite scales.
 *
 * Parity status of each function is pinned by tests under tests/ against
 * brute force, closed forms, hand-worked examples and library routines
 * (numpy.lexsort, numpy.packbits, numpy.random.Philox).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define BCO_F32 0
#define BCO_F16 1

/* ------------------------------------------------------------------ */
/* Sizes                                                                */
/* ------------------------------------------------------------------ */

/* Parts-per-million form of a compression ratio; 0 means invalid. */
static uint64_t ratio_ppm(double ratio)
{
    if (!(ratio > 0.0) || ratio > 1.0) return 0;
    return (uint64_t)llround(ratio * 1e6);
}

/* k rule (reading of the paper's "1% compression rate", Sec. 5.1):
 * k = min(n, max(1, ceil(n * ratio))) with ratio taken in whole parts per
 * million so the ceiling is exact integer arithmetic; k = 0 when n = 0. */
uint64_t bco_k(uint64_t n, double ratio)
{
    uint64_t ppm = ratio_ppm(ratio);
    if (n == 0 || ppm == 0) return 0;
    uint64_t k = (n * ppm + 999999u) / 1000000u;
    if (k < 1) k = 1;
    if (k > n) k = n;
    return k;
}

/* Number of 32-bit words holding n sign bits (one bit per element). */
uint64_t bco_words(uint64_t n) { return (n + 31u) / 32u; }

/* ------------------------------------------------------------------ */
/* Element access                                                       */
/* ------------------------------------------------------------------ */

/* IEEE 754 binary16 -> binary32, written from the format definition:
 * value = (-1)^s * 2^(e-15) * 1.m for 0 < e < 31, (-1)^s * 2^-14 * 0.m for
 * e = 0 (subnormals, kept exactly), infinities and NaN for e = 31. */
float bco_f16_to_f32(uint16_t h)
{
    uint32_t s = (uint32_t)(h >> 15) & 1u;
    uint32_t e = (uint32_t)(h >> 10) & 31u;
    uint32_t m = (uint32_t)h & 1023u;
    float mag;
    if (e == 0) {
        mag = (float)m * 5.9604644775390625e-8f; /* m * 2^-24, exact */
    } else if (e == 31) {
        mag = m ? NAN : INFINITY;
    } else {
        mag = ldexpf((float)(1024u + m), (int)e - 25); /* 1.m * 2^(e-15) */
    }
    return s ? -mag : mag;
}

static float grad_at(const void* g, int dtype, uint64_t i)
{
    if (dtype == BCO_F16) return bco_f16_to_f32(((const uint16_t*)g)[i]);
    return ((const float*)g)[i];
}

static uint32_t f2u(float x) { uint32_t u; memcpy(&u, &x, 4); return u; }
static float u2f(uint32_t u) { float x; memcpy(&x, &u, 4); return x; }

/* Error-feedback accumulate (paper Sec. 2.3: compression is combined with
 * error feedback; Sec. 5.1: applied to every compression): the vector that
 * is compressed is v = g + e_old, one fp32 addition per element.  With no
 * residual (error feedback off) v = g. */
static float* ef_accumulate(const void* g, int dtype, const float* e_in, uint64_t n)
{
    float* v = (float*)malloc((n ? n : 1) * sizeof(float));
    if (!v) return NULL;
    for (uint64_t i = 0; i < n; ++i) {
        float gi = grad_at(g, dtype, i);
        v[i] = e_in ? gi + e_in[i] : gi;
    }
    return v;
}

/* Selection key: the magnitude bits of v as an unsigned integer.  For
 * finite values this orders by |v|; +0.0 and -0.0 tie. */
static uint32_t key_of(float x) { return f2u(x) & 0x7FFFFFFFu; }

/* ------------------------------------------------------------------ */
/* Top-k sparsification (paper Sec. 2.3; DGC at 1% in Sec. 5.1)         */
/* ------------------------------------------------------------------ */

typedef struct { uint32_t key; uint32_t idx; } kv_t;

/* Order used for selection: larger key first, lower index first on ties. */
static int cmp_key_desc_idx_asc(const void* a, const void* b)
{
    const kv_t* x = (const kv_t*)a;
    const kv_t* y = (const kv_t*)b;
    if (x->key != y->key) return x->key > y->key ? -1 : 1;
    if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;
    return 0;
}

static int cmp_u32_asc(const void* a, const void* b)
{
    uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
    return (x > y) - (x < y);
}

/* Write the sparse payload for the chosen index set and the residual.
 * Payload: indices ascending, values v[idx] unscaled.  Residual: what was
 * not transmitted, e_new = v with the transmitted entries set to +0.0. */
static void emit_sparse(const float* v, uint64_t n, uint32_t* sel, uint64_t k,
                        uint32_t* idx, float* val, float* e_out)
{
    qsort(sel, (size_t)k, sizeof(uint32_t), cmp_u32_asc);
    for (uint64_t j = 0; j < k; ++j) {
        idx[j] = sel[j];
        val[j] = v[sel[j]];
    }
    if (e_out) {
        for (uint64_t i = 0; i < n; ++i) e_out[i] = v[i];
        for (uint64_t j = 0; j < k; ++j) e_out[sel[j]] = 0.0f;
    }
}

/* Exact top-k: the first k indices of the order (key desc, index asc),
 * found by sorting all n entries. */
int bco_compress_topk(const void* g, int dtype, const float* e_in, uint64_t n,
                      uint64_t k, uint32_t* idx, float* val, float* e_out)
{
    if (k > n) return -1;
    float* v = ef_accumulate(g, dtype, e_in, n);
    kv_t* a = (kv_t*)malloc((n ? n : 1) * sizeof(kv_t));
    uint32_t* sel = (uint32_t*)malloc((k ? k : 1) * sizeof(uint32_t));
    if (!v || !a || !sel) { free(v); free(a); free(sel); return -2; }
    for (uint64_t i = 0; i < n; ++i) { a[i].key = key_of(v[i]); a[i].idx = (uint32_t)i; }
    qsort(a, (size_t)n, sizeof(kv_t), cmp_key_desc_idx_asc);
    for (uint64_t j = 0; j < k; ++j) sel[j] = a[j].idx;
    emit_sparse(v, n, sel, k, idx, val, e_out);
    free(v); free(a); free(sel);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11), from its published */
/* definition: four 64-bit counter words, two 64-bit key words, ten      */
/* rounds; each round multiplies counter words 0 and 2 by the two round  */
/* multipliers into 128-bit products, permutes and xors the halves with  */
/* the other counter words and the key; the key advances by the two      */
/* Weyl constants between rounds.                                         */
/* ------------------------------------------------------------------ */

#define PHILOX_M0 0xD2E7470EE14C6C93ull
#define PHILOX_M1 0xCA5A826395121157ull
#define PHILOX_W0 0x9E3779B97F4A7C15ull
#define PHILOX_W1 0xBB67AE8584CAA73Bull

void bco_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { k0 += PHILOX_W0; k1 += PHILOX_W1; }
        unsigned __int128 p0 = (unsigned __int128)PHILOX_M0 * c0;
        unsigned __int128 p1 = (unsigned __int128)PHILOX_M1 * c2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t n0 = hi1 ^ c1 ^ k0;
        uint64_t n1 = lo1;
        uint64_t n2 = hi0 ^ c3 ^ k1;
        uint64_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Random-stream identifiers (second key word). */
#define STREAM_RANDK 0u
#define STREAM_SAMPLE 1u

/* ------------------------------------------------------------------ */
/* Random-k (Randomk at 1% in paper Sec. 5.1)                            */
/*                                                                      */
/* Reading: k distinct indices drawn without replacement.  They are the */
/* images of 0..k-1 under a keyed pseudorandom permutation of [0, n):   */
/* a balanced four-round Feistel network on b-bit integers (b = the     */
/* bit length of n-1, at least 2, rounded up to even) restricted to     */
/* [0, n) by cycle-walking (Black and Rogaway, CT-RSA 2002).  The four  */
/* round keys come from one Philox4x64-10 block keyed by (seed, stream  */
/* 0) at counter (tensor_id, 0, 0, 0).  The round function is the       */
/* "lowbias32" integer hash (C. Wellons, hash-prospector) of the right  */
/* half xor the round key, masked to b/2 bits.                          */
/* ------------------------------------------------------------------ */

static uint32_t lowbias32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

/* Half-width h of the Feistel domain for a tensor of n elements. */
uint32_t bco_feistel_half_bits(uint64_t n)
{
    uint32_t b = 0;
    uint64_t m = n > 1 ? n - 1 : 0;
    while (m) { ++b; m >>= 1; }
    if (b < 2) b = 2;
    if (b & 1u) ++b;
    return b / 2;
}

void bco_randk_round_keys(uint64_t seed, uint32_t tensor_id, uint32_t rk[4])
{
    uint64_t ctr[4] = { tensor_id, 0, 0, 0 };
    uint64_t key[2] = { seed, STREAM_RANDK };
    uint64_t w[4];
    bco_philox4x64_10(ctr, key, w);
    for (int r = 0; r < 4; ++r) rk[r] = (uint32_t)w[r] ^ (uint32_t)(w[r] >> 32);
}

/* One application of the four-round Feistel permutation E on [0, 2^(2h)). */
uint64_t bco_feistel_encrypt(uint64_t x, uint32_t h, const uint32_t rk[4])
{
    uint32_t mask = (h >= 32) ? 0xFFFFFFFFu : ((1u << h) - 1u);
    uint32_t L = (uint32_t)(x >> h) & mask;
    uint32_t R = (uint32_t)x & mask;
    for (int r = 0; r < 4; ++r) {
        uint32_t F = lowbias32(R ^ rk[r]) & mask;
        uint32_t nL = R;
        uint32_t nR = L ^ F;
        L = nL; R = nR;
    }
    return ((uint64_t)L << h) | R;
}

/* The j-th random-k index of a tensor: E applied to j, then again while
 * the result lies outside [0, n).  Terminates because j < n lies on the
 * same cycle of the permutation E. */
uint64_t bco_randk_index(uint64_t n, uint64_t seed, uint32_t tensor_id, uint64_t j)
{
    uint32_t rk[4];
    bco_randk_round_keys(seed, tensor_id, rk);
    uint32_t h = bco_feistel_half_bits(n);
    uint64_t x = bco_feistel_encrypt(j, h, rk);
    while (x >= n) x = bco_feistel_encrypt(x, h, rk);
    return x;
}

int bco_compress_randk(const void* g, int dtype, const float* e_in, uint64_t n,
                       uint64_t k, uint64_t seed, uint32_t tensor_id,
                       uint32_t* idx, float* val, float* e_out)
{
    if (k > n) return -1;
    float* v = ef_accumulate(g, dtype, e_in, n);
    uint32_t* sel = (uint32_t*)malloc((k ? k : 1) * sizeof(uint32_t));
    if (!v || !sel) { free(v); free(sel); return -2; }
    uint32_t rk[4];
    bco_randk_round_keys(seed, tensor_id, rk);
    uint32_t h = bco_feistel_half_bits(n);
    for (uint64_t j = 0; j < k; ++j) {
        uint64_t x = bco_feistel_encrypt(j, h, rk);
        while (x >= n) x = bco_feistel_encrypt(x, h, rk);
        sel[j] = (uint32_t)x;
    }
    emit_sparse(v, n, sel, k, idx, val, e_out);
    free(v); free(sel);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Sampled-threshold top-k (DGC at 1% in paper Sec. 5.1)                */
/*                                                                      */
/* Steps: draw a seeded sample of m = ceil(1% of n) positions (uniform, */
/* with replacement, from Philox4x64-10 keyed by (seed, stream 1) at    */
/* counters (tensor_id, block, 0, 0)); the threshold is the k_s-th      */
/* largest sample key, k_s = the k rule applied to m; candidates are    */
/* the entries whose key is at least the threshold; if there are at    */
/* least k candidates keep the first k of them in the selection order   */
/* (trim), otherwise add the best k - |C| of the other entries in that  */
/* order (top up).  Reading: trimming and topping up both use the exact */
/* selection order, so the result is exactly k entries.                 */
/* ------------------------------------------------------------------ */

uint64_t bco_sample_size(uint64_t n) { return n == 0 ? 0 : (n + 99u) / 100u; }

int bco_compress_topk_sampled(const void* g, int dtype, const float* e_in, uint64_t n,
                              uint64_t k, double ratio, uint64_t seed, uint32_t tensor_id,
                              uint32_t* idx, float* val, float* e_out,
                              uint64_t* n_candidates)
{
    if (k > n) return -1;
    float* v = ef_accumulate(g, dtype, e_in, n);
    uint64_t m = bco_sample_size(n);
    uint32_t* skey = (uint32_t*)malloc((m ? m : 1) * sizeof(uint32_t));
    kv_t* cand = (kv_t*)malloc((n ? n : 1) * sizeof(kv_t));
    kv_t* rest = (kv_t*)malloc((n ? n : 1) * sizeof(kv_t));
    uint32_t* sel = (uint32_t*)malloc((k ? k : 1) * sizeof(uint32_t));
    if (!v || !skey || !cand || !rest || !sel) {
        free(v); free(skey); free(cand); free(rest); free(sel); return -2;
    }
    /* 1. seeded sample of positions */
    for (uint64_t j = 0; j < m; j += 4) {
        uint64_t ctr[4] = { tensor_id, j / 4, 0, 0 };
        uint64_t key[2] = { seed, STREAM_SAMPLE };
        uint64_t w[4];
        bco_philox4x64_10(ctr, key, w);
        for (uint64_t q = 0; q < 4 && j + q < m; ++q) {
            uint64_t pos = (uint64_t)(((unsigned __int128)w[q] * n) >> 64);
            skey[j + q] = key_of(v[pos]);
        }
    }
    /* 2. threshold: k_s-th largest sample key */
    uint32_t thr = 0;
    if (m > 0) {
        uint64_t ks = bco_k(m, ratio);
        kv_t* s = (kv_t*)malloc(m * sizeof(kv_t));
        if (!s) { free(v); free(skey); free(cand); free(rest); free(sel); return -2; }
        for (uint64_t j = 0; j < m; ++j) { s[j].key = skey[j]; s[j].idx = (uint32_t)j; }
        qsort(s, (size_t)m, sizeof(kv_t), cmp_key_desc_idx_asc);
        thr = s[ks - 1].key;
        free(s);
    }
    /* 3. candidates (index order) and the rest */
    uint64_t nc = 0, nr = 0;
    for (uint64_t i = 0; i < n; ++i) {
        kv_t e; e.key = key_of(v[i]); e.idx = (uint32_t)i;
        if (e.key >= thr) cand[nc++] = e; else rest[nr++] = e;
    }
    if (n_candidates) *n_candidates = nc;
    /* 4. trim or top up to exactly k */
    qsort(cand, (size_t)nc, sizeof(kv_t), cmp_key_desc_idx_asc);
    if (nc >= k) {
        for (uint64_t j = 0; j < k; ++j) sel[j] = cand[j].idx;
    } else {
        qsort(rest, (size_t)nr, sizeof(kv_t), cmp_key_desc_idx_asc);
        for (uint64_t j = 0; j < nc; ++j) sel[j] = cand[j].idx;
        for (uint64_t j = nc; j < k; ++j) sel[j] = rest[j - nc].idx;
    }
    emit_sparse(v, n, sel, k, idx, val, e_out);
    free(v); free(skey); free(cand); free(rest); free(sel);
    return 0;
}

/* ------------------------------------------------------------------ */
/* One-bit sign quantization (EFSignSGD in paper Sec. 5.1; 1-bit        */
/* quantization in Sec. 2.3)                                            */
/*                                                                      */
/* Reading: the scale is the mean magnitude of the error-corrected      */
/* vector, s = (float)((sum_i |v_i| in fp64, index order) / n); the bit */
/* of element i is the IEEE sign bit of v_i (1 = negative, -0.0         */
/* included); word w holds elements 32w..32w+31, element i at bit       */
/* i mod 32, unused high bits zero.  Decoding gives -s for a set bit    */
/* and +s otherwise; the residual is e_new = v - decoded.               */
/* ------------------------------------------------------------------ */

int bco_compress_sign(const void* g, int dtype, const float* e_in, uint64_t n,
                      uint32_t* words, float* scale, float* e_out)
{
    float* v = ef_accumulate(g, dtype, e_in, n);
    if (!v) return -2;
    double sum = 0.0;
    for (uint64_t i = 0; i < n; ++i) sum += fabs((double)v[i]);
    float s = (n == 0) ? 0.0f : (float)(sum / (double)n);
    *scale = s;
    uint64_t nw = bco_words(n);
    for (uint64_t w = 0; w < nw; ++w) words[w] = 0u;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t bit = f2u(v[i]) >> 31;
        words[i / 32] |= bit << (i % 32);
    }
    if (e_out) {
        for (uint64_t i = 0; i < n; ++i) {
            uint32_t bit = f2u(v[i]) >> 31;
            float d = bit ? -s : s;
            e_out[i] = v[i] - d;
        }
    }
    free(v);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Residual update from a payload produced elsewhere:                   */
/* e_new = (g + e_old) - decompress(payload), elementwise in fp32.      */
/* ------------------------------------------------------------------ */

int bco_residual_update_sparse(const void* g, int dtype, float* e_inout, uint64_t n,
                               uint64_t k, const uint32_t* idx, const float* val)
{
    float* v = ef_accumulate(g, dtype, e_inout, n);
    float* dec = (float*)calloc(n ? n : 1, sizeof(float));
    if (!v || !dec) { free(v); free(dec); return -2; }
    for (uint64_t j = 0; j < k; ++j) {
        if (idx[j] >= n) { free(v); free(dec); return -1; }
        dec[idx[j]] = val[j];
    }
    for (uint64_t i = 0; i < n; ++i) e_inout[i] = v[i] - dec[i];
    free(v); free(dec);
    return 0;
}

int bco_residual_update_sign(const void* g, int dtype, float* e_inout, uint64_t n,
                             const uint32_t* words, float scale)
{
    float* v = ef_accumulate(g, dtype, e_inout, n);
    if (!v) return -2;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t bit = (words[i / 32] >> (i % 32)) & 1u;
        float d = bit ? -scale : scale;
        e_inout[i] = v[i] - d;
    }
    free(v);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Decompress and aggregate W payloads of one tensor (paper Sec. 3.1,   */
/* Reason #2: after gathering, each node decompresses the N compressed  */
/* tensors and aggregates them).                                        */
/*                                                                      */
/* Reading: aggregation is a sum scaled by alpha (alpha = 1 for a sum,  */
/* 1/W for a mean).  Sparse: each output element starts at +0.0 and     */
/* receives the workers' values in ascending worker order, one fp32     */
/* addition each, then alpha times that sum.  Sign: see below.          */
/* ------------------------------------------------------------------ */

int bco_aggregate_sparse(int W, uint64_t n, const uint32_t* const* idx_w,
                         const float* const* val_w, const uint64_t* k_w,
                         float alpha, float* out)
{
    float* acc = (float*)malloc((n ? n : 1) * sizeof(float));
    if (!acc) return -2;
    for (uint64_t i = 0; i < n; ++i) acc[i] = 0.0f;
    for (int w = 0; w < W; ++w) {
        for (uint64_t j = 0; j < k_w[w]; ++j) {
            uint32_t i = idx_w[w][j];
            if (i >= n) { free(acc); return -1; }
            acc[i] = acc[i] + val_w[w][j];
        }
    }
    for (uint64_t i = 0; i < n; ++i) out[i] = alpha * acc[i];
    free(acc);
    return 0;
}

/* Worker-ordered fp32 sum of the decoded sign values (each output starts at
 * +0.0 and adds the W values in ascending worker order).  Not the sign
 * aggregate's definition (bco_aggregate_sign below is); exported so that the
 * pins can bound the exact sum against a recursive summation. */
int bco_aggregate_sign_ordered(int W, uint64_t n, const uint32_t* const* words_w,
                               const float* scale_w, float alpha, float* out)
{
    for (uint64_t i = 0; i < n; ++i) {
        float acc = 0.0f;
        for (int w = 0; w < W; ++w) {
            uint32_t bit = (words_w[w][i / 32] >> (i % 32)) & 1u;
            float d = bit ? -scale_w[w] : scale_w[w];
            acc = acc + d;
        }
        out[i] = alpha * acc;
    }
    return 0;
}

/* Exact sum of fp32 terms in a 320-bit two's-complement fixed-point integer
 * whose unit is 2^-149 (the smallest fp32 subnormal), then one
 * round-to-nearest-even to fp32.  Finite terms only. */
typedef struct { uint64_t l[5]; } acc320_t;

static void acc_add_shifted(acc320_t* a, uint64_t m, int pos, int negative)
{
    /* t = m << pos as a 320-bit value */
    uint64_t t[5] = { 0, 0, 0, 0, 0 };
    int limb = pos / 64, sh = pos % 64;
    t[limb] = m << sh;
    if (sh && limb + 1 < 5) t[limb + 1] = m >> (64 - sh);
    if (negative) { /* two's complement of t */
        unsigned __int128 c = 1;
        for (int q = 0; q < 5; ++q) {
            c += (unsigned __int128)(~t[q]);
            t[q] = (uint64_t)c;
            c >>= 64;
        }
    }
    unsigned __int128 c = 0;
    for (int q = 0; q < 5; ++q) {
        c += (unsigned __int128)a->l[q] + t[q];
        a->l[q] = (uint64_t)c;
        c >>= 64;
    }
}

static void acc_add_f32(acc320_t* a, float x)
{
    uint32_t u = f2u(x);
    uint32_t e = (u >> 23) & 255u, f = u & 0x7FFFFFu;
    if (e == 0 && f == 0) return;
    uint64_t m = e ? (uint64_t)(f | 0x800000u) : (uint64_t)f;
    int pos = e ? (int)e - 1 : 0; /* value = m * 2^(pos - 149) */
    acc_add_shifted(a, m, pos, (int)(u >> 31));
}

static float acc_round_f32(const acc320_t* a)
{
    uint64_t v[5];
    int neg = (int)(a->l[4] >> 63);
    memcpy(v, a->l, sizeof v);
    if (neg) {
        unsigned __int128 c = 1;
        for (int q = 0; q < 5; ++q) {
            c += (unsigned __int128)(~v[q]);
            v[q] = (uint64_t)c;
            c >>= 64;
        }
    }
    int h = -1;
    for (int q = 4; q >= 0 && h < 0; --q)
        if (v[q]) h = q * 64 + 63 - __builtin_clzll(v[q]);
    if (h < 0) return 0.0f; /* exact zero rounds to +0.0 */
    float mag;
    if (h < 24) {
        mag = ldexpf((float)v[0], -149); /* fewer than 25 bits: exact */
    } else {
        /* 24 leading bits, the round bit below them, and a sticky bit */
        uint64_t mant = 0;
        for (int b = h; b > h - 24; --b) mant = (mant << 1) | ((v[b / 64] >> (b % 64)) & 1u);
        int rb = (int)((v[(h - 24) / 64] >> ((h - 24) % 64)) & 1u);
        int sticky = 0;
        for (int b = h - 25; b >= 0 && !sticky; --b) sticky = (int)((v[b / 64] >> (b % 64)) & 1u);
        if (rb && (sticky || (mant & 1u))) ++mant;
        mag = ldexpf((float)mant, h - 23 - 149);
    }
    return neg ? -mag : mag;
}

/* Order-free sum of the W decoded values of one element, the aggregate's
 * reading for the kinds whose decoded values are 0 or +-scale (sign,
 * TernGrad).  The paper only has every node decompress the gathered payloads
 * and sum them (Sec. 3.1, Reason #2); no addition order is given, so the sum
 * is the one every order of exact arithmetic reaches:
 *   - NaN when some decoded value is NaN, or when both +Inf and -Inf occur;
 *   - else +Inf or -Inf when an infinity occurs;
 *   - else the exact real sum of the finite values (subnormals included),
 *     rounded once to fp32 (round to nearest even; an exact zero gives +0.0,
 *     a sum beyond the fp32 range rounds to an infinity). */
typedef struct { acc320_t a; int nan, pinf, ninf; } xsum_t;

static void xsum_add(xsum_t* s, float d)
{
    if (isnan(d)) s->nan = 1;
    else if (isinf(d)) { if (d > 0.0f) s->pinf = 1; else s->ninf = 1; }
    else acc_add_f32(&s->a, d);
}

static float xsum_round(const xsum_t* s)
{
    if (s->nan || (s->pinf && s->ninf)) return NAN;
    if (s->pinf) return INFINITY;
    if (s->ninf) return -INFINITY;
    return acc_round_f32(&s->a);
}

/* Sign aggregate (reading): alpha times the order-free sum above of the W
 * decoded values d_w = (bit ? -s_w : +s_w), one fp32 multiplication. */
int bco_aggregate_sign(int W, uint64_t n, const uint32_t* const* words_w,
                       const float* scale_w, float alpha, float* out)
{
    for (uint64_t i = 0; i < n; ++i) {
        xsum_t s;
        memset(&s, 0, sizeof s);
        for (int w = 0; w < W; ++w) {
            uint32_t bit = (words_w[w][i / 32] >> (i % 32)) & 1u;
            xsum_add(&s, bit ? -scale_w[w] : scale_w[w]);
        }
        out[i] = alpha * xsum_round(&s);
    }
    return 0;
}

/* Exact sum of m fp32 values rounded once to fp32 (exported for pins). */
float bco_exact_sum_f32(const float* x, uint64_t m)
{
    acc320_t a;
    memset(&a, 0, sizeof a);
    for (uint64_t i = 0; i < m; ++i) acc_add_f32(&a, x[i]);
    return acc_round_f32(&a);
}

/* Bit pattern helpers exported for tests. */
uint32_t bco_f32_bits(float x) { return f2u(x); }
float bco_bits_f32(uint32_t u) { return u2f(u); }

/* ------------------------------------------------------------------ */
/* Stochastic b-bit quantization with error feedback (paper Sec. 2.3:   */
/* quantization maps fp32 gradients to fewer bits -- 8 bits, 2 bits     */
/* (TernGrad), 1 bit -- and is combined with error feedback).  The      */
/* paper defines none of these operators; the reading here follows the */
/* cited stochastic quantizers (TernGrad: ternary levels scaled by the  */
/* largest magnitude, each nonzero with probability |v|/max; QSGD:      */
/* s uniform levels with stochastic rounding to a neighbouring level),  */
/* with the largest magnitude as the norm so that the scale does not    */
/* depend on a summation order:                                         */
/*                                                                      */
/*   bits b in {2, 4, 8}; levels s = 2^(b-1) - 1 (1, 7, 127);           */
/*   v = fl32(g + e_old); m = max |v_i| (the payload's scale);          */
/*   inv = fl32(s / m) and unit = fl32(m / s), each one fp64 division   */
/*   rounded to fp32;                                                   */
/*   x_i = fl32(|v_i| * inv); if x_i >= s the level is s, else with     */
/*   l = floor(x_i) and p = x_i - l (exact), the level is l + 1 when    */
/*   U_i < p and l otherwise;                                           */
/*   U_i = (u_i >> 8) * 2^-24 with u_i the 32-bit word i mod 8 of the   */
/*   Philox4x64-10 block at counter (tensor_id, i / 8, 0, 0), key       */
/*   (seed, stream 2): 64-bit output word (i mod 8) / 2, its low half   */
/*   for even i, high half for odd i;                                   */
/*   code = 0 for level 0, else level | (sign bit of v_i) << (b - 1);   */
/*   codes are packed b bits each, LSB first, 32 / b per 32-bit word,   */
/*   each tensor starting a new word;                                   */
/*   decode: d = 0 for level 0, else +-fl32(level * unit) with the sign */
/*   of the code;  e_new = fl32(v - d);  m = 0 gives all-zero codes.    */
/* ------------------------------------------------------------------ */

#define STREAM_QUANT 2u

int bco_quant_levels(int bits)
{
    if (bits != 2 && bits != 4 && bits != 8) return 0;
    return (1 << (bits - 1)) - 1;
}

uint64_t bco_quant_words(uint64_t n, int bits) { return (n * (uint64_t)bits + 31u) / 32u; }

/* The uniform U_i of element i (exact fp32 in [0, 1)). */
float bco_quant_uniform(uint64_t seed, uint32_t tensor_id, uint64_t i)
{
    uint64_t ctr[4] = { tensor_id, i / 8u, 0, 0 };
    uint64_t key[2] = { seed, STREAM_QUANT };
    uint64_t w[4];
    bco_philox4x64_10(ctr, key, w);
    uint64_t x = w[(i % 8u) / 2u];
    uint32_t u = (i % 2u) ? (uint32_t)(x >> 32) : (uint32_t)x;
    return (float)(u >> 8) * 0x1p-24f;
}

/* Decoded value of one code for a tensor whose payload scale is m. */
float bco_quant_decode(uint32_t code, int bits, float m)
{
    int s = bco_quant_levels(bits);
    uint32_t level = code & ((1u << (bits - 1)) - 1u);
    if (level == 0 || s == 0) return 0.0f;
    float unit = (float)((double)m / (double)s);
    float mag = (float)level * unit;
    return ((code >> (bits - 1)) & 1u) ? -mag : mag;
}

static uint32_t quant_code_at(const uint32_t* words, uint64_t i, int bits)
{
    uint64_t pos = i * (uint64_t)bits;
    return (words[pos / 32u] >> (pos % 32u)) & ((1u << bits) - 1u);
}

int bco_compress_quant(const void* g, int dtype, const float* e_in, uint64_t n, int bits,
                       uint64_t seed, uint32_t tensor_id, uint32_t* words, float* scale,
                       float* e_out)
{
    int s = bco_quant_levels(bits);
    if (s == 0) return -1;
    float* v = ef_accumulate(g, dtype, e_in, n);
    if (!v) return -2;
    float m = 0.0f;
    for (uint64_t i = 0; i < n; ++i) {
        float a = fabsf(v[i]);
        if (a > m) m = a;
    }
    *scale = m;
    uint64_t nw = bco_quant_words(n, bits);
    for (uint64_t w = 0; w < nw; ++w) words[w] = 0u;
    float inv = m > 0.0f ? (float)((double)s / (double)m) : 0.0f;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t level = 0;
        if (m > 0.0f) {
            float x = fabsf(v[i]) * inv;
            if (x >= (float)s) {
                level = (uint32_t)s;
            } else {
                float l = floorf(x);
                float p = x - l;
                level = (uint32_t)l + (bco_quant_uniform(seed, tensor_id, i) < p ? 1u : 0u);
            }
        }
        uint32_t code = level ? (level | ((f2u(v[i]) >> 31) << (bits - 1))) : 0u;
        uint64_t pos = i * (uint64_t)bits;
        words[pos / 32u] |= code << (pos % 32u);
    }
    if (e_out) {
        for (uint64_t i = 0; i < n; ++i)
            e_out[i] = v[i] - bco_quant_decode(quant_code_at(words, i, bits), bits, m);
    }
    free(v);
    return 0;
}

int bco_residual_update_quant(const void* g, int dtype, float* e_inout, uint64_t n, int bits,
                              const uint32_t* words, float scale)
{
    if (bco_quant_levels(bits) == 0) return -1;
    float* v = ef_accumulate(g, dtype, e_inout, n);
    if (!v) return -2;
    for (uint64_t i = 0; i < n; ++i)
        e_inout[i] = v[i] - bco_quant_decode(quant_code_at(words, i, bits), bits, scale);
    free(v);
    return 0;
}

/* Quantizer aggregate: alpha * (sum over the workers of the decoded
 * values).  4- and 8-bit codes: each output starts at +0.0 and adds the W
 * decoded values in ascending worker order, one fp32 addition each.  2-bit
 * (TernGrad) codes decode to 0 or +-scale, as sign bits decode to +-scale,
 * and take the sign kind's reading: the order-free exact sum of the decoded
 * values rounded once (xsum above). */
int bco_aggregate_quant(int W, uint64_t n, int bits, const uint32_t* const* words_w,
                        const float* scale_w, float alpha, float* out)
{
    if (bco_quant_levels(bits) == 0) return -1;
    if (bits == 2) {
        for (uint64_t i = 0; i < n; ++i) {
            xsum_t s;
            memset(&s, 0, sizeof s);
            for (int w = 0; w < W; ++w)
                xsum_add(&s, bco_quant_decode(quant_code_at(words_w[w], i, bits), bits, scale_w[w]));
            out[i] = alpha * xsum_round(&s);
        }
        return 0;
    }
    for (uint64_t i = 0; i < n; ++i) {
        float acc = 0.0f;
        for (int w = 0; w < W; ++w)
            acc = acc + bco_quant_decode(quant_code_at(words_w[w], i, bits), bits, scale_w[w]);
        out[i] = alpha * acc;
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* DGC momentum correction and momentum-factor masking around a sparse  */
/* compression (DGC is the paper's sparsification operator, Sec. 5.1;   */
/* its momentum correction keeps a per-tensor velocity u next to the    */
/* accumulated gradient, which is the error-feedback residual here):    */
/*   u_new = fl32(fl32(m * u) + g);  the sparse kind then compresses    */
/*   u_new with the residual e (v = fl32(u_new + e), selection, payload, */
/*   e_new = v with the chosen entries +0.0);  masking sets u_new to    */
/*   +0.0 at the chosen entries as well.                                */
/* This function is the first step; the compression and the masking are */
/* the existing functions applied in that order (see the Python side).  */
/* ------------------------------------------------------------------ */

int bco_dgc_momentum(const void* g, int dtype, float* u_inout, uint64_t n, float m)
{
    for (uint64_t i = 0; i < n; ++i) {
        float mu = m * u_inout[i];
        u_inout[i] = mu + grad_at(g, dtype, i);
    }
    return 0;
}

/* DGC local gradient clipping (DGC's clipping before the gradient joins
 * the accumulation; a reading of it, the paper naming DGC only as its
 * sparsifier, Sec. 5.1): over the T gradients of one step, the L2 norm
 * ||g|| = sqrt(sum of widen(g_i)^2), each square exact in fp64, summed in
 * fp64 in tensor order then index order, the square root in fp64;
 * factor c = fl32(clip / ||g||) when ||g|| > clip, else exactly 1. */
float bco_dgc_clip_factor(int T, const void* const* g, const int* dtype, const uint64_t* n, double clip)
{
    double s = 0.0;
    for (int t = 0; t < T; ++t)
        for (uint64_t i = 0; i < n[t]; ++i) {
            const double x = (double)grad_at(g[t], dtype[t], i);
            s += x * x;
        }
    const double norm = sqrt(s);
    return norm > clip ? (float)(clip / norm) : 1.0f;
}

/* The velocity step with the clipped gradient: u = fl32(fl32(m u) +
 * fl32(c g)) (c = 1 leaves g unchanged, so the step is bco_dgc_momentum's). */
int bco_dgc_momentum_clipped(const void* g, int dtype, float* u_inout, uint64_t n, float m, float c)
{
    for (uint64_t i = 0; i < n; ++i) {
        float mu = m * u_inout[i];
        float gc = c * grad_at(g, dtype, i);
        u_inout[i] = mu + gc;
    }
    return 0;
}
