/*
 * precog.h -- C ABI of libprecog: the PRECOG hot path on one MI355X (gfx950).
 *
 * PRECOG (arXiv 2608.02560) encodes each corpus chunk once into the final
 * recurrent state of a gated selective SSM, stores that state, and at query
 * time retrieves the best-matching state by cosine similarity, injects it as
 * the initial state and runs only the query tokens (Sec. 4.2).  Theorem 1
 * (Sec. 4.3) makes the injection exact: S(h0, c ++ q) = S(S(h0, c), q).
 *
 * The three operations of that path are exported here:
 *   precog_scan_encode      selective-SSM prefill scan with injectable h0 and
 *                           captured hT (Eq. 1, Sec. 3; capture, Sec. 4.2)
 *   precog_retrieve_top1    exact cosine top-1 over a key index (Sec. 4.2)
 *   precog_inject_gather    h0[q] <- store[idx[q]] (Sec. 4.2, query time)
 * for callers that cannot allocate device memory:
 *   precog_retrieve_top1_noalloc  top-1 with a fixed library-held workspace
 * with the injection fused into the query prefill:
 *   precog_scan_encode_indexed  the scan starting from store[idx] rows or
 *                           their top-k softmax composition
 * the SMC trajectory variant of the scan and the complex-A scan:
 *   precog_scan_trajectory  the scan keeping every k-th state (Sec. 5.1-5.2)
 *   precog_scan_complex     Eq. 1 with a diagonal complex A (Sec. 3)
 * the top-k extension of retrieval and injection:
 *   precog_retrieve_topk    exact top-k with scores (Sec. 4.4, Fig. 1)
 *   precog_retrieve_prepare / precog_retrieve_topk_prepared
 *                           the same retrieval over an index prepared once
 *   precog_inject_compose   softmax-weighted composition of the top-k states
 *                           (Sec. 5.4 Eq. smc-fusion)
 *   precog_inject_fuse      the same over an episodic and a corpus store, plus
 *                           the session's semantic state (Sec. 5.4)
 * and the memory-consolidation steps of SMC:
 *   precog_smc_route        two-stage cluster routing (Sec. 5.1)
 *   precog_smc_consolidate  semantic-state EMA (Sec. 5.3 Eq. smc-ema)
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are device pointers owned by the caller.  The
 *     library never allocates, frees, copies between host and device, or
 *     synchronises; work is enqueued on `stream` (a hipStream_t passed as
 *     void*, NULL = the default stream) and runs asynchronously.
 *   - Arguments are validated on the host before anything is enqueued.  On a
 *     validation failure nothing is written and the status says why.  A HIP
 *     launch failure returns PRECOG_ERR_HIP.  No C++ exception crosses the
 *     ABI.  The only library state is a per-device cache of the architecture
 *     check and, for precog_retrieve_top1_noalloc, a fixed device array per
 *     device with its looked-up address.
 *   - Layouts are row-major with the last index fastest.
 *   - Entry points may be called concurrently from several host threads on
 *     different streams; calls on one stream execute in order.
 */
#ifndef PRECOG_H
#define PRECOG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PRECOG_F32 = 0,  /* IEEE binary32 */
    PRECOG_BF16 = 1, /* bfloat16 (upper half of binary32) */
    PRECOG_F16 = 2   /* IEEE binary16 */
} precog_dtype;

typedef enum {
    PRECOG_OK = 0,
    PRECOG_ERR_NULL = 1,      /* a required pointer is NULL */
    PRECOG_ERR_SHAPE = 2,     /* negative size, unsupported N, E, ... */
    PRECOG_ERR_DTYPE = 3,     /* dtype not supported for that tensor */
    PRECOG_ERR_STRIDE = 4,    /* state batch stride smaller than D*N */
    PRECOG_ERR_ALIGN = 5,     /* pointer or size breaks the alignment rule */
    PRECOG_ERR_WORKSPACE = 6, /* workspace missing or too small */
    PRECOG_ERR_ARCH = 7,      /* current device is not gfx950 */
    PRECOG_ERR_HIP = 8        /* a HIP runtime call or launch failed */
} precog_status;

/* ------------------------------------------------------------------------ */
/* Selective-SSM prefill scan                                               */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t batch;  /* B: independent sequences (corpus chunks or queries) */
    int64_t seqlen; /* L: tokens per sequence, >= 0 */
    int64_t dim;    /* D: channels, a multiple of 8 */
    int64_t dstate; /* N: state size per channel, one of 1,2,4,8,16,32,64 */
    precog_dtype in_dtype;    /* x, dt, B, C, z: PRECOG_F32 or PRECOG_BF16 */
    precog_dtype out_dtype;   /* y: PRECOG_F32 or PRECOG_BF16 */
    precog_dtype state_dtype; /* h0 and hT storage: PRECOG_F32 or PRECOG_F16;
                                 the running state is always fp32 */
    int64_t h0_batch_stride;  /* elements between batch rows of h0; 0 = D*N */
    int64_t hT_batch_stride;  /* elements between batch rows of hT; 0 = D*N
                                 (e.g. layers*D*N to land each final state
                                 in its layer slot of a [chunks, layers, D, N]
                                 store) */
    int64_t chunk;            /* time-chunk length of the two-level scan:
                                 0 = chosen by the library; >= L = one pass */
} precog_scan_desc;

/* Bytes of device workspace precog_scan_encode needs for `desc` (0 when the
 * scan runs in one pass).  Returns 0 for an invalid descriptor too; the
 * encode call reports the error. */
size_t precog_scan_workspace_bytes(const precog_scan_desc *desc);

/* The recurrence of Eq. 1 (Sec. 3) with a real, positive diagonal A, rolled
 * over each sequence from h0 (the rollout S(h0, x_1:L) of App. A):
 *
 *   h_t[d,n] = exp(-dt_t[d] * A[d,n]) * h_{t-1}[d,n] + B_t[n] * x_t[d] * dt_t[d]
 *   y_t[d]   = (sum_n C_t[n] h_t[d,n] + Dskip[d] x_t[d]) * silu(z_t[d])
 *   hT       = h_L   (the state after the last token; offline indexing
 *                     captures it, Sec. 4.2)
 *
 * with silu(v) = v / (1 + exp(-v)) and t = 1..L per batch row.  Arguments:
 *   x, dt, z   [B, L, D] in desc->in_dtype.  dt > 0 (already a timescale;
 *              no softplus is applied).  z NULL = no gate (factor 1).
 *   A          [D, N] fp32, A > 0 (decay < 1: the stable SSM of App. A).
 *   B, C       [B, L, N] in desc->in_dtype, shared by all channels.
 *   Dskip      [D] fp32; NULL = no skip term.
 *   h0         state rows in desc->state_dtype, row b at h0 + b*stride, each
 *              row [D, N]; NULL = zero initial state.
 *   y          [B, L, D] in desc->out_dtype; NULL = state-only encode (then C,
 *              z and Dskip are not read and may be NULL).
 *   hT         state rows like h0 (its own stride); NULL = not captured.
 *              hT may alias h0 exactly (in-place streaming prefill: the
 *              state of one call becomes the injected state of the next).
 *   workspace  device memory of precog_scan_workspace_bytes(desc) bytes,
 *              16-byte aligned (NULL allowed when that size is 0).
 * Alignment: every tensor base pointer 16-byte aligned, D % 8 == 0, state
 * strides % 8 == 0.  y must not overlap any input.  Results are
 * deterministic: the same inputs give bitwise the same outputs. */
precog_status precog_scan_encode(const precog_scan_desc *desc, const void *x,
                                 const void *dt, const float *A, const void *B,
                                 const void *C, const void *z,
                                 const float *Dskip, const void *h0, void *y,
                                 void *hT, void *workspace,
                                 size_t workspace_bytes, void *stream);

/* precog_scan_encode whose initial states come straight from a state store:
 * the query-time injection (Sec. 4.2) fused into the prefill, so the
 * injected states are never written out and read back.
 *
 *   h0 of batch row b = store row h0_idx[b]                    (h0_score NULL)
 *   h0 of batch row b = sum_j w_j store[h0_idx[b*k + j]]       (h0_score given)
 *
 * the second with w = softmax(h0_score[b*k .. b*k+k-1] / tau), exactly as
 * precog_inject_compose forms it (Sec. 5.4 Eq. smc-fusion).
 *
 * Arguments as precog_scan_encode, with h0 replaced by:
 *   store       state rows in desc->state_dtype, row r at store + r*stride
 *               (stride = desc->h0_batch_stride, 0 = D*N), each row [D, N];
 *               a layer of a multi-layer store is addressed by offsetting
 *               `store` and setting the stride to the row pitch.
 *   store_rows  rows of the store (>= 0).
 *   h0_idx      [B, k] int32, device memory, 16-byte aligned.  An index
 *               outside [0, store_rows) reads nothing and starts that batch
 *               row from NaN (as the gather and the composition write NaN).
 *   h0_score    [B, k] fp64 retrieval scores (precog_retrieve_topk), 16-byte
 *               aligned, or NULL for the plain gather (then k must be 1).
 *   k, tau      rows composed per batch row, 1..64, and the softmax
 *               temperature, tau > 0 (unused without scores).
 * The arithmetic is exactly that of precog_inject_gather (or
 * precog_inject_compose) into a state of desc->state_dtype followed by
 * precog_scan_encode: the results are bitwise those of the two calls.  hT
 * must not overlap the store.  NULL h0_idx with work to do is
 * PRECOG_ERR_NULL; store may be NULL only when store_rows is 0; k or tau out
 * of range is PRECOG_ERR_SHAPE. */
precog_status precog_scan_encode_indexed(const precog_scan_desc *desc, const void *x,
                                         const void *dt, const float *A, const void *B,
                                         const void *C, const void *z,
                                         const float *Dskip, const void *store,
                                         int64_t store_rows, const int32_t *h0_idx,
                                         const double *h0_score, int64_t k, double tau,
                                         void *y, void *hT, void *workspace,
                                         size_t workspace_bytes, void *stream);

/* precog_scan_encode that also keeps the thinned state trajectory of the SMC
 * encode (Sec. 5.1 Eq. smc-trajectory, the fidelity dial of Sec. 5.2):
 *
 *   traj[b, s, d, n] = h_t[d, n]  for t = every * (s + 1), s = 0..L/every - 1
 *
 * i.e. the state after every `every`-th token (t counted from 1).  every = 1
 * keeps the whole trajectory (K = N_c), every = L only the final state
 * (K = 1, equal to hT).  All other arguments and outputs are exactly those of
 * precog_scan_encode (y and hT may be NULL; a state-only trajectory encode
 * reads x, dt and B only).
 *   traj   [B, L / every, D, N] in desc->state_dtype (fp16 rounds to nearest
 *          even), 16-byte aligned; NULL only when L < every (nothing is
 *          captured then).
 *   every  >= 1, else PRECOG_ERR_SHAPE. */
precog_status precog_scan_trajectory(const precog_scan_desc *desc,
                                     const void *x, const void *dt,
                                     const float *A, const void *B,
                                     const void *C, const void *z,
                                     const float *Dskip, const void *h0,
                                     void *y, void *hT, void *traj,
                                     int64_t every, void *workspace,
                                     size_t workspace_bytes, void *stream);

/* The scan with the diagonal complex A of Sec. 3 (Eq. 1 with A_k = a_k +
 * i w_k; the paper's frequencies are w_k = pi k, its real part is the
 * negative of a here, see precog_scan_encode):
 *
 *   h_t[d,n] = exp(-dt_t[d] (A_re[d,n] + i A_im[d,n])) h_{t-1}[d,n]
 *              + B_t[n] x_t[d] dt_t[d]                       (complex state)
 *   y_t[d]   = (sum_n C_t[n] Re h_t[d,n] + Dskip[d] x_t[d]) * silu(z_t[d])
 *
 * Arguments as precog_scan_encode, except:
 *   A_re, A_im  [D, N] fp32; A_re > 0.
 *   h0, hT      complex state rows [D, N, 2] ((real, imaginary) interleaved)
 *               in desc->state_dtype; batch strides in elements, 0 = 2*D*N.
 *   desc->dstate in {1, 2, 4, 8, 16}.
 *   Time chunks as in precog_scan_encode (desc->chunk, 0 = automatic: one
 *               pass when batch x channels fill the GPU; chunks are capped
 *               so that chunk * max(D, N) * 4 < 2^31).  A chunked scan folds
 *               the chunks' end states with the product of their decays,
 *               exp(-(A_re + i A_im) sum dt) (its angle reduced in fp64),
 *               and replays each chunk from its carried-in state.
 *   workspace   precog_scan_complex_workspace_bytes(desc) bytes (0 for one
 *               pass: NULL allowed), 16-byte aligned; about
 *               B * chunks * D * (8 N + 4) bytes.
 * The rotation uses the hardware sine and cosine of the angle reduced to
 * [0, 1) revolutions; the magnitude uses the hardware exp2. */
size_t precog_scan_complex_workspace_bytes(const precog_scan_desc *desc);

precog_status precog_scan_complex(const precog_scan_desc *desc, const void *x,
                                  const void *dt, const float *A_re,
                                  const float *A_im, const void *B,
                                  const void *C, const void *z,
                                  const float *Dskip, const void *h0, void *y,
                                  void *hT, void *workspace,
                                  size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* Cosine top-1 retrieval                                                   */
/* ------------------------------------------------------------------------ */

/* Bytes of device workspace precog_retrieve_top1 needs for (Q, M, E). */
size_t precog_retrieve_workspace_bytes(int64_t Q, int64_t M, int64_t E);

/* Query-time retrieval of Sec. 4.2: for each query q,
 *   idx[q] = argmax_i <query[q], index[i]>
 * over the M key rows, the cosine similarity for unit-norm rows.  The result
 * is exact: it equals the argmax of the fp64 inner products summed in index
 * order (products of fp32 values are exact in fp64), ties going to the
 * lowest row.  A matrix-core screen (queries and keys rounded to
 * fp16(2^8 v), exact products summed in fp32) proposes candidates within a
 * proven error margin and only those are rescored in fp64 (a lone candidate
 * needs none; several are ordered by an fp64 tree sum when its proven error
 * separates them, else by the sequential fp64 sums).  Non-finite inputs give
 * unspecified indices.
 *   query_emb  [Q, E] fp32     index_emb [M, E] fp32 (rows of any norm;
 *              the margin scales with the row norms; a query or key of norm
 *              245 or more could overflow the fp16 operands, and then every
 *              key is rescored: exact, but as slow as a full fp64 search)
 *   idx        [Q] int32 output; M == 0 gives -1
 *   E % 4 == 0, 4 <= E <= 4096; pointers 16-byte aligned.
 *   workspace  precog_retrieve_workspace_bytes(Q, M, E) bytes, 16-byte
 *              aligned, about 9 Q M / 32 + 4 M bytes (per query and
 *              32-key block the screen keeps its largest score, that key
 *              and the second largest);
 *              ceil(M / 32) * ceil(Q / 128) must not exceed 2^31 - 1. */
precog_status precog_retrieve_top1(const float *query_emb,
                                   const float *index_emb, int64_t Q, int64_t M,
                                   int64_t E, int32_t *idx, void *workspace,
                                   size_t workspace_bytes, void *stream);

/* Top-k retrieval (the top-k extension of Sec. 4.4 and Fig. 1): for each
 * query q, idx[q, 0..k-1] are the k rows with the largest inner products,
 * best first, ordered exactly as by the fp64 scores of precog_retrieve_top1
 * (inner products summed in index order, products exact), ties to the
 * lower row; score[q, j] is the fp64 score of idx[q, j].  The same screen
 * and proven margin as precog_retrieve_top1, with the k-th largest block
 * maximum in place of the maximum, so the result is exact.
 *   query_emb [Q, E] fp32    index_emb [M, E] fp32
 *   k         1 <= k <= 64 and k <= M, else PRECOG_ERR_SHAPE
 *   idx       [Q, k] int32 output
 *   score     [Q, k] fp64 output, or NULL
 *   E % 4 == 0, 4 <= E <= 4096; pointers 16-byte aligned.
 *   workspace precog_retrieve_workspace_bytes(Q, M, E) bytes (the same as
 *             for top-1).  Non-finite inputs give unspecified indices. */
/* Bytes of the device array behind precog_retrieve_top1_noalloc: 32 MiB,
 * held on each device the library runs on until the process ends. */
#define PRECOG_NOALLOC_SCRATCH_BYTES (32u << 20)

/* precog_retrieve_top1 for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments (minus the workspace), same result, bit for
 * bit; its workspace is a fixed array of PRECOG_NOALLOC_SCRATCH_BYTES in
 * this library's device memory, one per device.  The call allocates
 * nothing (no hipMalloc, hipFree or allocating library routine); its first
 * call on a device looks up that device's copy of the array.
 *   Limit: precog_retrieve_workspace_bytes(Q, M, E) must not exceed
 *   PRECOG_NOALLOC_SCRATCH_BYTES (about Q * M <= 1.1e8 pairs), else
 *   PRECOG_ERR_WORKSPACE and nothing is enqueued.
 *   Every call on one device shares that device's array: calls that overlap
 *   on one device (different streams without ordering between them, or
 *   several host threads) race and give unspecified indices.  Calls ordered
 *   on one stream are safe; nothing carries over from one call to the next. */
precog_status precog_retrieve_top1_noalloc(const float *query_emb,
                                           const float *index_emb, int64_t Q,
                                           int64_t M, int64_t E, int32_t *idx,
                                           void *stream);

precog_status precog_retrieve_topk(const float *query_emb,
                                   const float *index_emb, int64_t Q, int64_t M,
                                   int64_t E, int64_t k, int32_t *idx,
                                   double *score, void *workspace,
                                   size_t workspace_bytes, void *stream);

/* Prepared index (the offline side of Sec. 4.2: keys are embedded once).
 * Bytes of the prepared form of an [M, E] key index: the keys' fp16(2^8 k)
 * screen operands in the screen's own tile order, their squared norms and
 * the largest squared norm of every 32-key block.  0 for M < 1 or an E the
 * retrieval calls reject. */
size_t precog_retrieve_index_bytes(int64_t M, int64_t E);

/* Writes the prepared form of index_emb ([M, E] fp32, the same rows the
 * retrieval calls read) into `prepared` (device memory, caller-owned,
 * precog_retrieve_index_bytes(M, E) bytes, 16-byte aligned).  Asynchronous
 * on `stream`; the prepared form stays valid while index_emb is unchanged.
 *   1 <= M < 2^31, 4 <= E <= 4096, E % 4 == 0, else PRECOG_ERR_SHAPE /
 *   PRECOG_ERR_ALIGN; too small a buffer gives PRECOG_ERR_WORKSPACE. */
precog_status precog_retrieve_prepare(const float *index_emb, int64_t M,
                                      int64_t E, void *prepared,
                                      size_t prepared_bytes, void *stream);

/* precog_retrieve_topk (and, with k = 1 and score NULL, precog_retrieve_top1)
 * with the screen reading the prepared operands and norms instead of
 * converting index_emb on every call.  Results are identical to the
 * unprepared calls: the same operands, the same margin, the same fp64
 * decision over index_emb's fp32 rows (which must be the rows `prepared`
 * was made from).  Arguments as precog_retrieve_topk, plus
 *   prepared   from precog_retrieve_prepare(index_emb, M, E, ...), 16-byte
 *              aligned, prepared_bytes >= precog_retrieve_index_bytes(M, E)
 *              (else PRECOG_ERR_WORKSPACE; NULL gives PRECOG_ERR_NULL). */
precog_status precog_retrieve_topk_prepared(const float *query_emb,
                                            const float *index_emb,
                                            const void *prepared,
                                            size_t prepared_bytes, int64_t Q,
                                            int64_t M, int64_t E, int64_t k,
                                            int32_t *idx, double *score,
                                            void *workspace,
                                            size_t workspace_bytes,
                                            void *stream);

/* The whole query-time path of Sec. 4.2 in one call: the exact top-1
 * retrieval, the injection of the retrieved state and the query prefill
 * from it (Eq. 1; Theorem 1 of Sec. 4.3 is why the prefill from the stored
 * state equals processing chunk and query together):
 *   idx[b] = the top-1 of precog_retrieve_top1 (or, with `prepared`, of
 *            precog_retrieve_topk_prepared with k = 1) for query_emb row b,
 *   then exactly precog_scan_encode_indexed(desc, x, dt, A, B, C, z, Dskip,
 *            state_store, M, idx, NULL, 1, 1.0, y, hT, ...).
 * idx, y and hT are bitwise those of the two calls.  Batch row b of the scan
 * is query b (desc->batch = Q); the store has one state row per key of the
 * index (M rows of [D, N] at stride desc->h0_batch_stride, 0 = D*N, in
 * desc->state_dtype).  With N = 16, bf16 inputs, one pass over time (the
 * automatic chunking picks one when batch x channels fill the GPU, or
 * desc->chunk >= L) and y with a gate (or y NULL), each prefill workgroup
 * decides its own query in one wave while the other waves fetch their first
 * tokens, then starts from the decided row (one launch for the decision,
 * injection and prefill); otherwise the retrieval's decision and the
 * prefill run as two launches.
 *   query_emb  [Q, E] fp32    index_emb [M, E] fp32 (as precog_retrieve_top1)
 *   prepared   NULL, or the prepared index of index_emb (precog_retrieve_prepare)
 *              with prepared_bytes >= precog_retrieve_index_bytes(M, E)
 *              (else PRECOG_ERR_WORKSPACE)
 *   state_store  [M, D, N] rows as above; NULL only when M == 0
 *   idx        [Q] int32 output (M == 0 gives -1 and NaN start states)
 *   x ... hT   as precog_scan_encode
 *   workspace  precog_query_workspace_bytes(desc, M, E) bytes, 16-byte aligned.
 * Every argument of both halves is validated before anything is launched;
 * the status codes are those of the two calls. */
size_t precog_query_workspace_bytes(const precog_scan_desc *desc, int64_t M, int64_t E);
precog_status precog_query_top1_prefill(const precog_scan_desc *desc,
                                        const float *query_emb,
                                        const float *index_emb,
                                        const void *prepared,
                                        size_t prepared_bytes, int64_t M,
                                        int64_t E, const void *state_store,
                                        int32_t *idx, const void *x,
                                        const void *dt, const float *A,
                                        const void *B, const void *C,
                                        const void *z, const float *Dskip,
                                        void *y, void *hT, void *workspace,
                                        size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* State injection                                                          */
/* ------------------------------------------------------------------------ */

/* The injection of Sec. 4.2, h_init <- h^(i*): copies state rows of S
 * elements (e.g. D*N for one layer, layers*D*N for a whole model state)
 *   h0[q, :] = store[idx[q], :]     for q = 0..Q-1
 * from store [M, S] (store_dtype F32 or F16) into h0 [Q, S] (h0_dtype F32 or
 * F16; F16 -> F32 widens exactly, F32 -> F16 rounds to nearest even).
 * An idx outside [0, M) fills that row of h0 with NaN and reads nothing.
 * S % 8 == 0; pointers 16-byte aligned. */
precog_status precog_inject_gather(const void *state_store,
                                   precog_dtype store_dtype, int64_t M,
                                   int64_t S, const int32_t *idx, int64_t Q,
                                   void *h0, precog_dtype h0_dtype,
                                   void *stream);

/* Top-k injection (Sec. 5.4 Eq. smc-fusion, the composition of Fig. 1):
 *   h0[q, :] = sum_{j<k} w_j store[idx[q, j], :],
 *   w_j = exp(score[q, j] / tau) / sum_i exp(score[q, i] / tau)
 * The paper's softmax has no temperature: tau = 1 is that formula; other
 * tau > 0 scale the logits.  Weights are formed in fp64 and rounded once to
 * fp32; the sum runs in fp32 in rank order (j = 0 first), one fused
 * multiply-add per term, so each element is within (k + 2) 2^-24
 * sum_j w_j |h_j| of the exact value (before an fp16 output's rounding).
 * k = 1 reproduces precog_inject_gather bit for bit.
 *   store   [M, S] F32 | F16     h0 [Q, S] F32 | F16 (RNE when F16)
 *   idx     [Q, k] int32 (e.g. from precog_retrieve_topk); a row with any
 *           index outside [0, M) is filled with NaN
 *   score   [Q, k] fp64, finite
 *   1 <= k <= 64; tau > 0 and finite; S % 8 == 0; pointers 16-byte aligned */
precog_status precog_inject_compose(const void *state_store,
                                    precog_dtype store_dtype, int64_t M,
                                    int64_t S, const int32_t *idx,
                                    const double *score, int64_t Q, int64_t k,
                                    double tau, void *h0, precog_dtype h0_dtype,
                                    void *stream);

/* ------------------------------------------------------------------------ */
/* Structured Memory Consolidation (Sec. 5)                                 */
/* ------------------------------------------------------------------------ */

/* Joint retrieval at query time (Sec. 5.4, Eq. smc-fusion): the candidates
 * of the session's episodic store and of the corpus, each from its own exact
 * top-k (precog_retrieve_topk over its own key index with the same query
 * embedding), are ranked together by score -- larger first; equal scores:
 * episodic before corpus, then the lower row, then the earlier list entry --
 * and the k best are composed as in precog_inject_compose, plus the
 * session's semantic state s with weight lambda (the paper adds it as a
 * baseline term and gives no weight; lambda = 1 adds it as is, 0 leaves it
 * out):
 *   h0[q] = sum_{j<k} w_j h^(j) + lambda * semantic[semantic_row[q]],
 *   w = softmax(score / tau) over the k selected scores.
 *   episodic_store [episodic_rows, S], corpus_store [corpus_rows, S] and
 *              semantic [semantic_rows, S]: store_dtype (F32 | F16)
 *   episodic_idx / episodic_score  [Q, episodic_k] int32 / fp64
 *   corpus_idx / corpus_score      [Q, corpus_k] int32 / fp64
 *              (episodic_k, corpus_k in 0..64; either list may be empty)
 *   k          1..64, k <= episodic_k + corpus_k
 *   semantic   NULL: no baseline term (semantic_row, lambda unread);
 *              semantic_row [Q] int32, e.g. the flat sub-cluster that
 *              precog_smc_route returned for the session
 *   h0         [Q, S] output in h0_dtype (F32 | F16, RNE)
 *   S % 8 == 0; tau > 0 finite; lambda finite; pointers 16-byte aligned.
 * Arithmetic: the weights as precog_inject_compose forms them (fp64, rounded
 * once to fp32), then one fp32 fma per term in rank order and one for the
 * semantic term.  With an empty corpus list and no semantic state the result
 * equals precog_inject_compose's bit for bit.  A candidate or semantic row
 * outside its store gives a NaN row. */
precog_status precog_inject_fuse(const void *episodic_store,
                                 int64_t episodic_rows,
                                 const int32_t *episodic_idx,
                                 const double *episodic_score,
                                 int64_t episodic_k, const void *corpus_store,
                                 int64_t corpus_rows,
                                 const int32_t *corpus_idx,
                                 const double *corpus_score, int64_t corpus_k,
                                 precog_dtype store_dtype, int64_t S, int64_t Q,
                                 int64_t k, double tau, const void *semantic,
                                 const int32_t *semantic_row,
                                 int64_t semantic_rows, double lambda,
                                 void *h0, precog_dtype h0_dtype,
                                 void *stream);

/* Two-stage routing of Sec. 5.1 (Eqs. smc-domain, smc-sub) for C chunk
 * embeddings phi(c):
 *   domain_out[c] = m* = argmax_m <phi(c), p_m>
 *   sub_out[c]    = j* = argmax_j <phi(c), q_{m*, j}>
 *   flat_out[c]   = m* * n_sub + j* (the row of the sub-cluster's semantic
 *                   state in an [n_domains * n_sub, S] table; NULL = skip)
 * Scores are exact: fp64 sums of the exact products, in feature order;
 * equal scores go to the lower index.  Non-finite inputs give unspecified
 * (in-range) routes.
 *   emb          [C, E] fp32     domain_protos [n_domains, E] fp32
 *   sub_protos   [n_domains, n_sub, E] fp32
 *   1 <= n_domains, n_sub <= 64; E % 4 == 0, 4 <= E <= 4096; outputs int32
 *   [C]; pointers 16-byte aligned. */
precog_status precog_smc_route(const float *emb, int64_t C, int64_t E,
                               const float *domain_protos, int64_t n_domains,
                               const float *sub_protos, int64_t n_sub,
                               int32_t *domain_out, int32_t *sub_out,
                               int32_t *flat_out, void *stream);

/* Semantic consolidation of Sec. 5.3 (Eq. smc-ema), applied in chunk order:
 *   for c = 0..C-1:  states[target[c]] <- (1 - alpha) states[target[c]]
 *                                         + alpha contrib[c]
 * in place, e.g. with target = flat_out of precog_smc_route and contrib =
 * the chunks' final states (their K = 1 contributions).  A target outside
 * [0, R) leaves every state unchanged for that chunk.  Each update is one
 * fp32 fused multiply-add with alpha and 1 - alpha rounded once to fp32
 * (alpha = 1 replaces the state exactly); F16 states are rounded to nearest
 * even after every update, as separate calls would.
 *   states   [R, S] F32 | F16, updated in place (R <= 65535)
 *   contrib  [C, S] F32 | F16; must not overlap states
 *   target   [C] int32
 *   0 < alpha <= 1; S % 8 == 0; pointers 16-byte aligned */
precog_status precog_smc_consolidate(void *states, precog_dtype state_dtype,
                                     int64_t R, int64_t S, const void *contrib,
                                     precog_dtype contrib_dtype,
                                     const int32_t *target, int64_t C,
                                     double alpha, void *stream);

/* Static, human-readable name of a status code. */
const char *precog_status_string(precog_status s);

#ifdef __cplusplus
}
#endif

#endif /* PRECOG_H */
