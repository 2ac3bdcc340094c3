/*
 * bytecomp_oracle_omp.c -- the CPU oracle run on every host core, for the
 * benchmark's CPU baseline.
 *
 * TEST INFRASTRUCTURE ONLY, like bytecomp_oracle.c, whose functions this
 * file includes unchanged.  It adds list-level entry points that run those
 * same per-tensor functions in parallel with OpenMP: compression over the
 * tensors of a list (each tensor on one thread), aggregation over the
 * tensors and, within a tensor, over ranges of 4096 elements.  Every output
 * element is computed by exactly the serial code on the same inputs, so the
 * results are bit-identical to the serial oracle at any thread count (a CPU
 * test checks this).  No arithmetic is changed or tuned.
 *
 * Kinds: 0 top-k, 1 sampled top-k, 2 random-k, 3 sign, 4 TernGrad (2-bit),
 * 5 QSGD 4-bit, 6 QSGD 8-bit.
 */
#include "bytecomp_oracle.c"

#include <omp.h>

int bco_omp_max_threads(void) { return omp_get_max_threads(); }

/* First position p in [0, k) with ix[p] >= x (k if none); ix ascending. */
static uint64_t first_at_least(const uint32_t* ix, uint64_t k, uint64_t x)
{
    uint64_t a = 0, b = k;
    while (a < b) {
        uint64_t mid = a + (b - a) / 2;
        if ((uint64_t)ix[mid] < x) a = mid + 1; else b = mid;
    }
    return a;
}

static int quant_bits_of(int kind) { return kind == 4 ? 2 : kind == 5 ? 4 : kind == 6 ? 8 : 0; }

/* Compress T tensors.  g[t], dtype[t], e_in[t] (may be NULL), n[t],
 * tensor_id[t]; outputs at per-tensor offsets: sparse kinds idx/val at
 * off[t] entries, word kinds words at off[t] words and scale[t]; e_out[t]
 * (may be NULL) receives the new residual.  Returns 0 or the first nonzero
 * per-tensor status. */
int bco_compress_list(int kind, int T, const void* const* g, const int* dtype, const float* const* e_in,
                      const uint64_t* n, const uint32_t* tensor_id, double ratio, uint64_t seed,
                      const uint64_t* off, uint32_t* idx, float* val, uint32_t* words, float* scale,
                      float* const* e_out, int threads)
{
    int rc_all = 0;
#pragma omp parallel for schedule(dynamic, 1) num_threads(threads) reduction(| : rc_all)
    for (int t = 0; t < T; ++t) {
        int rc = 0;
        const uint64_t k = bco_k(n[t], ratio);
        switch (kind) {
            case 0:
                rc = bco_compress_topk(g[t], dtype[t], e_in[t], n[t], k, idx + off[t], val + off[t], e_out[t]);
                break;
            case 1: {
                uint64_t nc = 0;
                rc = bco_compress_topk_sampled(g[t], dtype[t], e_in[t], n[t], k, ratio, seed, tensor_id[t],
                                               idx + off[t], val + off[t], e_out[t], &nc);
                break;
            }
            case 2:
                rc = bco_compress_randk(g[t], dtype[t], e_in[t], n[t], k, seed, tensor_id[t], idx + off[t],
                                        val + off[t], e_out[t]);
                break;
            case 3:
                rc = bco_compress_sign(g[t], dtype[t], e_in[t], n[t], words + off[t], scale + t, e_out[t]);
                break;
            default:
                rc = bco_compress_quant(g[t], dtype[t], e_in[t], n[t], quant_bits_of(kind), seed, tensor_id[t],
                                        words + off[t], scale + t, e_out[t]);
                break;
        }
        rc_all |= rc ? 1 : 0;
    }
    return rc_all ? -1 : 0;
}

/* Aggregate T tensors of W payloads.  a_w[w] / b_w[w]: worker w's arrays
 * (sparse: idx, val at off[t]; word kinds: words at off[t], scales b_w[w][t]
 * as floats); out[t] receives n[t] floats.  Work items are (tensor, range
 * of 4096 elements); a range runs the serial function on its slice: words
 * from the range's first word, sparse entries of the range rebased. */
int bco_aggregate_list(int kind, int W, int T, const uint64_t* n, const uint64_t* off,
                       const void* const* a_w, const void* const* b_w, float alpha, float* const* out,
                       int threads)
{
    const uint64_t R = 4096;
    uint64_t* item0 = (uint64_t*)malloc(((size_t)T + 1) * sizeof(uint64_t));
    if (!item0) return -2;
    item0[0] = 0;
    for (int t = 0; t < T; ++t) item0[t + 1] = item0[t] + (n[t] + R - 1) / R;
    const int64_t items = (int64_t)item0[T];
    int rc_all = 0;
#pragma omp parallel num_threads(threads) reduction(| : rc_all)
    {
        const uint32_t** pa = (const uint32_t**)malloc(((size_t)W + 1) * sizeof(void*));
        const float** pb = (const float**)malloc(((size_t)W + 1) * sizeof(void*));
        uint64_t* kk = (uint64_t*)malloc(((size_t)W + 1) * sizeof(uint64_t));
        float* sc = (float*)malloc(((size_t)W + 1) * sizeof(float));
        uint32_t** rebased = (uint32_t**)calloc((size_t)W + 1, sizeof(uint32_t*));
        if (!pa || !pb || !kk || !sc || !rebased) rc_all |= 1;
#pragma omp for schedule(dynamic, 4)
        for (int64_t it = 0; it < items; ++it) {
            if (!pa || !pb || !kk || !sc || !rebased) continue;
            int t = 0;
            while (item0[t + 1] <= (uint64_t)it) ++t;
            const uint64_t lo = ((uint64_t)it - item0[t]) * R;
            const uint64_t m = n[t] - lo < R ? n[t] - lo : R;
            int rc = 0;
            if (kind <= 2) {
                for (int w = 0; w < W; ++w) {
                    const uint32_t* ix = (const uint32_t*)a_w[w] + off[t];
                    const uint64_t kt = off[t + 1] - off[t];
                    const uint64_t p0 = first_at_least(ix, kt, lo), p1 = first_at_least(ix, kt, lo + m);
                    rebased[w] = (uint32_t*)malloc(((p1 - p0) ? (p1 - p0) : 1) * sizeof(uint32_t));
                    if (!rebased[w]) { rc = -2; continue; }
                    for (uint64_t q = p0; q < p1; ++q) rebased[w][q - p0] = ix[q] - (uint32_t)lo;
                    pa[w] = rebased[w];
                    pb[w] = (const float*)b_w[w] + off[t] + p0;
                    kk[w] = p1 - p0;
                }
                if (!rc) rc = bco_aggregate_sparse(W, m, pa, pb, kk, alpha, out[t] + lo);
                for (int w = 0; w < W; ++w) { free(rebased[w]); rebased[w] = NULL; }
            } else {
                const int bits = kind == 3 ? 1 : quant_bits_of(kind);
                for (int w = 0; w < W; ++w) {
                    pa[w] = (const uint32_t*)a_w[w] + off[t] + lo * (uint64_t)bits / 32u;
                    sc[w] = ((const float*)b_w[w])[t];
                }
                rc = kind == 3 ? bco_aggregate_sign(W, m, pa, sc, alpha, out[t] + lo)
                               : bco_aggregate_quant(W, m, bits, pa, sc, alpha, out[t] + lo);
            }
            rc_all |= rc ? 1 : 0;
        }
        free(pa); free(pb); free(kk); free(sc); free(rebased);
    }
    free(item0);
    return rc_all ? -1 : 0;
}
