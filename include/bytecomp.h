/*
 * bytecomp.h -- C ABI of the MI355X (gfx950) gradient-compression library.
 *
 * The library implements the per-tensor compression pipeline of ByteComp
 * (arXiv 2205.14465): compress each gradient tensor with error feedback,
 * exchange the payloads, then decompress and aggregate the N gathered
 * payloads (paper Sec. 3.1, Reason #2, indivisible scheme; Table "eight
 * action tasks": Comp, Comm_comp, Decomp).  The exchange itself is the
 * caller's: this library compresses, aggregates, and updates residuals.
 *
 * Operators (paper Sec. 5.1, "Compression algorithms"; Sec. 2.3):
 *   BC_TOPK          exact top-k sparsification
 *   BC_TOPK_SAMPLED  DGC-style top-k: threshold from a seeded sample, then
 *                    trimmed or topped up to exactly k (same result as
 *                    BC_TOPK, different cost)
 *   BC_RANDK         seeded random-k (Randomk)
 *   BC_SIGN1         1-bit sign with one scale per tensor (EFSignSGD)
 *   BC_TERNGRAD      2-bit stochastic ternary quantization (TernGrad)
 *   BC_QSGD4         4-bit stochastic quantization, 7 levels (QSGD)
 *   BC_QSGD8         8-bit stochastic quantization, 127 levels (QSGD)
 *                    (Sec. 2.3 names 8-bit, 2-bit and 1-bit quantization;
 *                    the paper does not evaluate the first two)
 * Error feedback (paper Sec. 2.3 and Sec. 5.1): the compressed vector is
 * v = g + e_old and the residual e_new = v - decompress(payload) is written
 * back in place.
 *
 * Conventions for every entry point:
 *   - Pointers named "device" must be device memory of the current HIP
 *     device; pointers named "host" are read before the call returns.
 *   - All work is enqueued on `stream` (a hipStream_t, NULL = the null
 *     stream); calls return without synchronising, with one exception: a
 *     descriptor-cache miss that evicts a table used from several streams
 *     waits for the device (below).  Argument errors are
 *     detected on the host before anything is enqueued: the call then
 *     returns a negative status and has no side effect.  Faults inside
 *     kernels surface at the caller's next synchronisation; with the
 *     environment variable BYTECOMP_DEBUG=1 every call synchronises and
 *     checks.
 *   - The caller owns every buffer.  The library keeps a small cache of
 *     per-device descriptor tables, reused while a call's tensor list is
 *     unchanged, and nothing else.  A call whose table is not cached
 *     allocates device and pinned host memory for it (hipMalloc,
 *     hipHostMalloc) when the evicted slot is too small, and first waits
 *     for the queued kernels that still read the evicted table: its event
 *     when one stream used it, the whole device when several did.  Callers
 *     that must not allocate use bytecomp_compress_noalloc.
 *   - Sizes: 0 <= n < 2^32 elements per tensor (indices are uint32);
 *     0 < ratio <= 1 with at least one part per million; T >= 0 (T = 0 is
 *     a no-op); W >= 1.
 *   - Alignment: fp32 gradients, residuals and aggregate outputs must be
 *     16-byte aligned; fp16 gradients 8-byte aligned (BC_E_ALIGN otherwise).
 *   - No C++ exception crosses this interface.
 */
#ifndef BYTECOMP_H
#define BYTECOMP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum bc_kind { BC_TOPK = 0, BC_TOPK_SAMPLED = 1, BC_RANDK = 2, BC_SIGN1 = 3,
               BC_TERNGRAD = 4, BC_QSGD4 = 5, BC_QSGD8 = 6 };
enum bc_dtype { BC_F32 = 0, BC_F16 = 1 };

enum bc_status {
    BC_OK = 0,
    BC_E_NULL = -1,       /* a required pointer is NULL                       */
    BC_E_KIND = -2,       /* unknown kind                                     */
    BC_E_DTYPE = -3,      /* unknown gradient dtype                           */
    BC_E_RATIO = -4,      /* ratio outside (0, 1] or below one part per million */
    BC_E_SIZE = -5,       /* a tensor has 2^32 or more elements, or a call is
                             beyond a kind's limits (see bytecomp_compress)   */
    BC_E_COUNT = -6,      /* T < 0, W < 1, or too many tensors/workers        */
    BC_E_WORKSPACE = -7,  /* workspace NULL or smaller than required          */
    BC_E_HIP = -8,        /* a HIP runtime call failed                        */
    BC_E_ALIGN = -9,      /* a dense buffer violates the alignment rule       */
    BC_E_DEVICE = -10     /* a kernel reported a failure (see bytecomp_device_status) */
};

/* One gradient tensor to compress.
 *   grad      device, n elements of `dtype`, read only
 *   residual  device, n fp32 error-feedback values, updated in place;
 *             NULL turns error feedback off (v = g, nothing written back)
 *   n         element count
 *   dtype     BC_F32 or BC_F16
 *   tensor_id key of the per-tensor random streams (BC_RANDK, the sample
 *             of BC_TOPK_SAMPLED, the rounding of the quantizers); by
 *             convention the tensor's position in
 *             the model, kept stable when only a subset is compressed */
typedef struct bc_tensor {
    const void* grad;
    float* residual;
    uint64_t n;
    uint32_t dtype;
    uint32_t tensor_id;
} bc_tensor;

/* One worker's payload for a list of T tensors, all device pointers.
 * Sparse kinds use idx/val: tensor t occupies entries [off[t], off[t+1])
 * (off from bytecomp_layout), indices tensor-local, strictly ascending,
 * values fp32.  BC_SIGN1 uses bits/scale: tensor t occupies words
 * [off[t], off[t+1]), element i of the tensor at bit (i mod 32) of word
 * off[t] + i/32 (1 = negative), bits past the tensor's end zero, and
 * scale[t] is its fp32 scale.  The quantizers (b = 2, 4, 8 bits per
 * element) also use bits/scale: element i's b-bit code at bit (i*b mod 32)
 * of word off[t] + i*b/32, codes past the tensor's end zero, scale[t] the
 * tensor's largest |v|.  Unused members may be NULL. */
typedef struct bc_payload {
    uint32_t* idx;
    float* val;
    uint32_t* bits;
    float* scale;
} bc_payload;

/* Human-readable text for a status code (static storage). */
const char* bytecomp_strerror(int status);

/* Payload layout (host only, no device work).
 * Sparse kinds: off[t+1] - off[t] = k_t = min(n_t, max(1, ceil(n_t *
 * ratio))) (0 when n_t = 0), the ratio taken in whole parts per million;
 * this reads the paper's "1% compression rate" (Sec. 5.1) as an exact k.
 * BC_SIGN1: off[t+1] - off[t] = ceil(n_t / 32) words (ratio ignored).
 * Quantizers: ceil(n_t * b / 32) words, b = 2, 4 or 8 (ratio ignored).
 *   n    host, T element counts
 *   off  host, T+1 entries written, off[0] = 0 */
int bytecomp_layout(int kind, double ratio, const uint64_t* n, int T, uint64_t* off);

/* Bytes of device workspace that bytecomp_compress and
 * bytecomp_decompress_aggregate need for this tensor list (host only).
 * W is the aggregation fan-in (use 1 for compression only). */
int bytecomp_workspace_size(int kind, double ratio, const uint64_t* n, int T, int W,
                            size_t* bytes);

/* Zero a workspace (enqueued on `stream`).  A workspace must be zero
 * before its first use; every successful call leaves the counters it used
 * at zero again, so one initialisation suffices.  Re-initialise after a
 * call that failed inside a kernel.  Calls that share a workspace must be
 * ordered (one stream, or synchronised streams): they race otherwise. */
int bytecomp_workspace_init(void* ws, size_t ws_bytes, void* stream);

/* Compress T tensors with error feedback (paper Sec. 2.3, Sec. 5.1).
 *   kind, ratio  operator and compression rate (ratio used by the sparse
 *                kinds only)
 *   seed         key of the random streams (BC_RANDK, BC_TOPK_SAMPLED,
 *                the quantizers' rounding); vary it per iteration
 *   t            host, T tensor descriptors
 *   out          payload to write (device pointers), laid out as
 *                bytecomp_layout describes
 *   ws, ws_bytes device workspace of at least bytecomp_workspace_size
 * Results: BC_TOPK and BC_TOPK_SAMPLED select the k_t entries of largest
 * |v| (ties to the lower index); BC_RANDK selects k_t distinct indices
 * from a keyed permutation of [0, n_t); both emit indices ascending with
 * values v[idx]; the residual becomes v with the selected entries +0.0.
 * BC_SIGN1 emits the sign bits of v and scale s_t = mean |v| (summed in
 * fp64) rounded to fp32; the residual becomes v - (bit ? -s_t : +s_t).
 * Quantizers (b bits, s = 2^(b-1) - 1 levels): m_t = max |v| is the
 * scale; with inv = fl32(s / m_t) and x = fl32(|v_i| * inv), the level is s
 * when x >= s, else floor(x) + 1 when U_i < x - floor(x) and floor(x)
 * otherwise, where U_i = (u >> 8) * 2^-24 and u is 32-bit word i mod 8
 * (low half of 64-bit output word (i mod 8)/2 for even i, high half for odd
 * i) of the Philox4x64-10 block at counter (tensor_id, i/8, 0, 0) and key
 * (seed, 2); the code is the level with the sign bit of v_i at bit b-1 (0
 * for level 0); decoding gives +-fl32(level * fl32(m_t / s)) and the
 * residual becomes v - decoded.
 * Limits of BC_RANDK: fewer than 2^32 payload entries in the call and at
 * most 2^22 chunks of 4096 elements (about 1.7e10 elements); BC_E_SIZE
 * otherwise. */
int bytecomp_compress(int kind, double ratio, uint64_t seed, const bc_tensor* t, int T,
                      bc_payload out, void* ws, size_t ws_bytes, void* stream);

/* bytecomp_compress for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same kernels and results, with no workspace argument.
 * The call's workspace and its descriptor table live in a device array of
 * the library, 16 MiB per GPU, held by each GPU the library runs on until
 * the process ends; the descriptor table is written by kernel launches (no
 * host-to-device copy) and the call allocates nothing.  Every call on a GPU
 * shares that GPU's array: calls that overlap on one GPU (other streams or
 * threads) race, so order them.  BC_E_SIZE, before anything is enqueued,
 * when the call's compress workspace plus its table (48 bytes per tensor
 * and 4 per 4096 elements) exceed 16 MiB: for BC_TOPK and BC_TOPK_SAMPLED
 * that is about 2M elements per call (8 bytes per element of candidate
 * space), for BC_SIGN1 and the quantizers several hundred million.  Every
 * other argument, status and result is bytecomp_compress's. */
int bytecomp_compress_noalloc(int kind, double ratio, uint64_t seed, const bc_tensor* t, int T,
                              bc_payload out, void* stream);

/* One DGC step (DGC is the paper's sparsification operator, Sec. 5.1):
 * momentum correction, sparse compression with error feedback, and
 * momentum-factor masking.  For every tensor, with u its velocity:
 *   u <- fl32(fl32(momentum * u) + g)    (fp16 g widened exactly)
 *   the sparse kind compresses u with the tensor's residual e, exactly as
 *   bytecomp_compress with grad = u (fp32) and residual = e would
 *   (v = u + e, payload, e <- v with +0.0 at the chosen entries)
 *   u <- +0.0 at the chosen entries.
 *   kind      BC_TOPK, BC_TOPK_SAMPLED or BC_RANDK (BC_E_KIND otherwise)
 *   velocity  host array of T device pointers: n_t fp32 values each,
 *             16-byte aligned, updated in place (zero them before the
 *             first step); a tensor's velocity, gradient and residual
 *             must not overlap (the step reads and writes them in one pass)
 *   t         the tensors; every residual must be non-NULL (it is DGC's
 *             accumulated gradient)
 * Every other argument, the workspace and the limits are bytecomp_compress's.
 * All arguments are checked before any work is enqueued.  DGC's sparsity
 * warm-up is a schedule of `ratio` over iterations, chosen by the caller
 * per call. */
int bytecomp_compress_dgc(int kind, double ratio, uint64_t seed, float momentum, const bc_tensor* t,
                          float* const* velocity, int T, bc_payload out, void* ws, size_t ws_bytes,
                          void* stream);

/* One DGC step with DGC's local gradient clipping before the momentum
 * correction (a reading of DGC's clipping; the paper names DGC as its
 * sparsifier, Sec. 5.1).  Over the call's T gradients (the worker's whole
 * gradient when the call holds it):
 *   norm = sqrt(sum over every element of widen(g)^2), each square exact
 *          in fp64, the sum in fp64 (per-chunk sums added in a fixed
 *          order, which differs from index order by the rounding of fp64
 *          additions only), the root in fp64
 *   c    = fl32(clip_norm / norm) if norm > clip_norm, else 1
 *   u   <- fl32(fl32(momentum * u) + fl32(c * g)), then the steps of
 *          bytecomp_compress_dgc (c = 1 gives its result bit for bit).
 *   clip_norm    the threshold (DGC scales its global threshold by
 *                N^(-1/2) for N workers; the caller passes the scaled
 *                value); >= 0, +inf never clips; BC_E_RATIO for a negative
 *                or NaN value
 *   clip_factor  device pointer to one float that receives c, or NULL
 * Every other argument and status is bytecomp_compress_dgc's. */
int bytecomp_compress_dgc_clip(int kind, double ratio, uint64_t seed, float momentum, double clip_norm,
                               const bc_tensor* t, float* const* velocity, int T, bc_payload out,
                               float* clip_factor, void* ws, size_t ws_bytes, void* stream);

/* Decompress W workers' payloads and aggregate them (paper Sec. 3.1,
 * Reason #2: each node decompresses the gathered payloads and aggregates
 * them; the aggregation is not an Allreduce because compressed
 * aggregation is not associative, Sec. 4.2.1, Dimension 3).
 *   in     host array of W payloads (device pointers), same layout for all
 *   n      host, T element counts
 *   out    host array of T device pointers to dense fp32 outputs
 *          (16-byte aligned)
 *   alpha  scale applied to each sum (1 = sum, 1/W = mean)
 *   ws     workspace: BC_SIGN1 and BC_TERNGRAD need bytecomp_workspace_size
 *          bytes (they keep a form and lookup tables per tensor there); the
 *          other kinds need its 256-byte header
 * Sparse kinds: out_t[i] = alpha * (sum over workers w = 0..W-1, in that
 * order, of worker w's value at i), each addition in fp32 starting from
 * +0.0; elements no worker sent are alpha * 0.
 * BC_SIGN1: out_t[i] = alpha * X(d_0,i, ..., d_W-1,i), d_w,i = -s_w,t if
 * worker w's bit i is set, else +s_w,t, where X is the sum every order of
 * exact arithmetic reaches: NaN if some d is NaN or both +Inf and -Inf
 * occur, else +-Inf if an infinity occurs, else the exact real sum of the
 * d rounded once to fp32 (nearest, ties to even; an exact zero gives +0.0;
 * past the fp32 range, an infinity).  This holds for every scale set
 * (subnormal, negative, widely spread or non-finite scales included).
 * BC_QSGD4, BC_QSGD8: out_t[i] = alpha * (sum over w = 0..W-1, in that
 * order, of worker w's decoded value at i), each addition in fp32 starting
 * from +0.0.  BC_TERNGRAD (decoded values 0 or +-s_w,t): alpha * X of the
 * decoded values, as for BC_SIGN1.  Quantizers: at most 1024 workers
 * (BC_E_COUNT otherwise).
 * Results are deterministic. */
int bytecomp_decompress_aggregate(int kind, double ratio, const bc_payload* in, int W,
                                  const uint64_t* n, int T, float* const* out, float alpha,
                                  void* ws, size_t ws_bytes, void* stream);

/* Divisible scheme, packing (paper Sec. 3.1, Reason #2, with the alltoall
 * figure: a compressed tensor is partitioned into parts, and node j receives
 * part j from every node).  Parts are element ranges: part q of tensor t is
 * [bounds[t*(parts+1)+q], bounds[t*(parts+1)+q+1]), where bounds (host) run
 * from 0 to n_t, never decrease, and every inner bound is a multiple of 32.
 * This packs part j of one payload `in` (laid out as bytecomp_layout
 * describes) into `out`:
 *   sparse kinds: tensor by tensor, the entries whose index lies in the
 *     range, in payload order, with the index rebased to the range
 *     (index - start); out.idx / out.val need room for every entry of `in`
 *     in the worst case;
 *   BC_SIGN1 and the quantizers: tensor by tensor, the words that cover
 *     the range (the layout bytecomp_layout gives for the range lengths)
 *     and every tensor's scale.
 *   part_off  device, T + 1 uint64: the packed offset of each tensor's part
 *             (entries, or words), then the total.
 * BC_E_ALIGN if an inner bound is not a multiple of 32, BC_E_SIZE if bounds
 * do not run from 0 to n_t in order.  Stream-ordered like the rest. */
int bytecomp_pack_part(int kind, double ratio, const uint64_t* n, int T, bc_payload in, int parts,
                       const uint64_t* bounds, int j, bc_payload out, uint64_t* part_off, void* stream);

/* Divisible scheme, aggregation of one part (paper Sec. 3.1, Reason #2: the
 * node that receives part j from every node decompresses and aggregates the
 * parts; compressing the aggregate again is bytecomp_compress on the dense
 * slices, and the final decompress is bytecomp_decompress_aggregate with
 * W = 1 per part).
 *   in        host, W payloads packed by bytecomp_pack_part for the same part
 *   part_off  host array of W device pointers: each sender's part_off
 *             (sparse kinds; ignored for the word kinds)
 *   len       host, T range lengths of the part
 *   out       host, T device pointers to dense fp32 slices (16-byte aligned)
 * out_t[i] = alpha * the senders' values at i summed exactly as
 * bytecomp_decompress_aggregate defines it for the kind (worker-ordered fp32
 * for the sparse kinds and 4-/8-bit codes, the exact sum rounded once for
 * sign and TernGrad), so the parts of all nodes assemble the whole
 * aggregate bit for bit.  Sparse kinds take at most 64
 * senders (BC_E_COUNT otherwise).  ws: as bytecomp_decompress_aggregate for
 * the range lengths. */
int bytecomp_aggregate_part(int kind, double ratio, const bc_payload* in, const uint64_t* const* part_off,
                            int W, const uint64_t* len, int T, float* const* out, float alpha, void* ws,
                            size_t ws_bytes, void* stream);

/* Error-feedback update from a payload computed elsewhere (e.g. by a CPU
 * compressor, the paper's CPU offloading, Sec. 4.4.3):
 * residual <- (g + residual) - decompress(own), elementwise in fp32.
 * Every tensor must have a non-NULL residual. */
int bytecomp_residual_update(int kind, double ratio, const bc_tensor* t, int T,
                             bc_payload own, void* stream);

/* CPU compression (paper Sec. 4.4.3, CPU offloading: the compression of
 * some tensors runs on the host CPUs instead of the GPU; Sec. 4.3 profiles
 * every operation on both).  bytecomp_compress on host memory: every
 * pointer (gradients, residuals, payload arrays) is host memory, and the
 * call runs synchronously on up to `threads` CPU threads (<= 0: one per
 * hardware thread).  Kinds BC_TOPK, BC_TOPK_SAMPLED (computed as BC_TOPK:
 * the same result), BC_RANDK and BC_SIGN1; BC_E_KIND for the quantizers.
 * Payload layout and results are bytecomp_compress's, except that a sign
 * scale is its fp64 sum taken in another order of additions (the two
 * differ by at most the fp64 rounding of the sums, under 1e-6 relative;
 * the residual uses the scale this call produced).  Errors: the argument
 * checks of bytecomp_compress (no stream or device checks); BC_E_SIZE when
 * host memory for the selection runs out; BC_E_HIP for any other host
 * failure.  Nothing is written to the outputs on an argument error. */
int bytecomp_cpu_compress(int kind, double ratio, uint64_t seed, const bc_tensor* t, int T,
                          bc_payload out, int threads);

/* CPU decompress-and-aggregate (the CPU side of the same offloading):
 * bytecomp_decompress_aggregate on host memory (payloads and outputs host
 * pointers), synchronous, up to `threads` CPU threads; the same results,
 * bit for bit, for BC_TOPK, BC_TOPK_SAMPLED, BC_RANDK and BC_SIGN1
 * (BC_E_KIND otherwise); at most 1024 workers. */
int bytecomp_cpu_decompress_aggregate(int kind, double ratio, const bc_payload* in, int W,
                                      const uint64_t* n, int T, float* const* out, float alpha, int threads);

/* Decision algorithm, host only (paper Sec. 4.3, the timeline model of
 * "Expressing interactions"; Sec. 4.4.3, Algorithm 2 and the Theorem's
 * enumeration of prod(|G_i| + 1) offloading count vectors).  A job of T
 * tensors in backward order (index 0 computed first); option o of tensor
 * i (0 none, 1 GPU indivisible, 2 GPU divisible, 3 CPU indivisible, 4 CPU
 * divisible) has the steps stage_off[i*5+o] .. stage_off[i*5+o+1]-1 after
 * its computation (compute_us[i] on the GPU): stage_res[q] the resource
 * (0 GPU, 1 CPU, 2 PCIe link, 3 network) and stage_us[q] the duration.
 * Every resource serves one step at a time in order of release (earliest
 * release, then lower tensor index, then earlier step); a tensor's
 * computation is released when the previous tensor's computation ends,
 * each later step when its previous step ends.  All arrays host.
 * bytecomp_plan_simulate: *iteration_us = the end of the last step under
 * the options option[T].  BC_E_KIND for an option outside 0..4. */
int bytecomp_plan_simulate(int T, const double* compute_us, const uint64_t* stage_off, const int32_t* stage_res,
                           const double* stage_us, const int32_t* option, double* iteration_us);

/* Algorithm 2's exhaustive search: groups g = 0..G-1 of tensors compressed
 * on the GPU (option 1 or 2), members group_member[group_off[g] ..
 * group_off[g+1]-1] in offloading order; count vector U offloads the first
 * U[g] members of each group (option + 2).  Every vector is evaluated (on
 * up to `threads` host threads, <= 0: all), in the order where the last
 * group's count varies fastest; the result is the first vector that
 * improves on the best so far by more than eps_us (vector 0 first).
 * best_counts[G] receives it, *best_us its iteration time, *evals the
 * number of vectors.  BC_E_SIZE, with nothing evaluated, when the number
 * of vectors exceeds max_evals; BC_E_KIND when a member is not on a GPU
 * option. */
int bytecomp_plan_enumerate(int T, const double* compute_us, const uint64_t* stage_off, const int32_t* stage_res,
                            const double* stage_us, const int32_t* option, int G, const uint64_t* group_off,
                            const int32_t* group_member, uint64_t max_evals, double eps_us, int threads,
                            int32_t* best_counts, double* best_us, uint64_t* evals);

/* Read (synchronously, on `stream`) and clear the kernel failure flags a
 * workspace holds; *flags receives them (0 = none).  No kernel of this
 * version sets one (bit 0 is reserved). */
int bytecomp_device_status(void* ws, size_t ws_bytes, void* stream, uint32_t* flags);

/* Selection statistics of the last top-k compress call on this workspace
 * (BC_TOPK or BC_TOPK_SAMPLED; the call's kind, ratio and tensor sizes
 * given again, no other call on the workspace since, and the path choice of
 * bytecomp_set_topk_few_chunks unchanged), read synchronously on `stream`:
 *   candidates  entries the exact selection examined, summed over the
 *               tensors: those at or above each tensor's candidate
 *               threshold (the sampled threshold, or for BC_TOPK and after
 *               a fallback the bin of the k-th key); at least the sum of
 *               the k_t, at most the sum of the n_t
 *   fallbacks   tensors whose sampled threshold left fewer than k_t
 *               candidates, so that they took the exact histogram path
 *               (0 for BC_TOPK and on the few-chunk path)
 * For monitoring and tuning (DGC's sampling); results never depend on it.
 * BC_E_KIND for other kinds, BC_E_WORKSPACE when ws is smaller than the
 * call's workspace, other argument errors as bytecomp_workspace_size. */
int bytecomp_topk_stats(int kind, double ratio, const uint64_t* n, int T, const void* ws, size_t ws_bytes,
                        void* stream, uint64_t* candidates, uint32_t* fallbacks);

/* Wait limit of the one-pass compress kernels (BC_SIGN1 and the quantizers
 * when every tensor fits the GPU's resident grid), process-wide.  Their
 * workgroups defer each chunk's residual (and codes) until the tensor's
 * scale, which needs a partial result of every chunk, is known, and wait
 * for the other chunks' partials at most `microseconds`.  Past that (the
 * grid not wholly resident, e.g. beside other kernels) a waiting workgroup
 * computes the missing partials itself, bit-identical to their owners'
 * (the same fixed-order arithmetic), so the results are the same either
 * way, only later.  0 makes every such wait do so at once (for tests of
 * that path).  Default 200; BC_E_SIZE above 10 s. */
int bytecomp_set_wait_limit(uint32_t microseconds);

/* Path choice for top-k compression (both kinds), for tests and tuning:
 * calls of at most `chunks` 4096-element chunks in total take the
 * few-chunk path (five launches, exact selection, a look-back across
 * chunks), larger calls the general pipeline; both give the same result.
 * Default and maximum 2048 (BC_E_SIZE above); 0 sends every call to the
 * general pipeline.  Process-wide; takes effect at the next call. */
int bytecomp_set_topk_few_chunks(uint32_t chunks);

/* Instrumentation, not part of the method: for callers that measure one
 * kernel's own duration (benchmarks).  The next launch, by any call, of
 * the kernel named `kernel` ("aggregate_sign", "aggregate_sparse",
 * "randk_stream", "topk_compact", "topk_hist" (the histogram pass of the
 * few-chunk top-k path), "sign_onepass", "sign_pass1" (the first kernel of
 * the two-pass sign compress), "quant_onepass", "quant_pass1",
 * "aggregate_quant") records `start_event` when it begins and `stop_event`
 * when it ends (HIP events created by the caller, on the launch's stream);
 * the request is then cleared.  Both events NULL clears a pending request
 * and returns 1 if one was pending (the named kernel did not run since the
 * request), 0 otherwise.  BC_E_KIND for an unknown name.  One request is
 * held at a time, process-wide. */
int bytecomp_time_next_launch(const char* kernel, void* start_event, void* stop_event);

#ifdef __cplusplus
}
#endif

#endif /* BYTECOMP_H */
