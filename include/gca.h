/*
 * libgca -- Grouped Cross Attention (GCA) hot path for AMD Instinct MI355X (gfx950).
 *
 * Method: "Efficient Length-Generalizable Attention via Causal Retrieval for
 * Long-Context Language Modeling" (arXiv 2410.01651), Methodology / Model
 * Architecture: causal relevance scores and top-k retrieval (Eq. 1), grouped
 * cross attention fused by the softmaxed scores (Eq. 2 and Eq. 3), and the
 * hardware-aware forward and backward passes of Appendix B (Algorithms 1-2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are DEVICE pointers, row-major and densely packed, in the
 *   layouts stated per argument.  The caller owns every buffer; the library never
 *   allocates, frees or retains memory.  Temporary storage comes from a caller
 *   workspace sized by gca_workspace_size().
 * - Chunks are numbered from 0.  In CAUSAL mode a sequence of L = n_chunks * S
 *   tokens has n_chunks chunks; landmark row t retrieves among chunks [0, t)
 *   (Eq. 1 ranges over strictly earlier chunks) and its retrieved set feeds the
 *   tokens of chunk t+1 (Eq. 2 applies C_t to chunk t+1).  In DECODE mode one new
 *   chunk of S tokens has one landmark query, scored against all n_chunks past
 *   chunks; that set feeds the new chunk's own tokens.
 * - nQ (landmark query rows) = n_chunks in CAUSAL mode and 1 in DECODE mode;
 *   Lq (query tokens) = nQ * Sq with Sq = S (S + 1 under GCA_FLAG_LMK_ROW);
 *   Lkv (key/value tokens) = n_chunks * S.  Query chunk c is rows
 *   [c * Sq, (c + 1) * Sq) of the query-side tensors.
 * - Retrieval heads: Hr = 1 shares one score per chunk pair across all H heads
 *   (Eq. 1 yields one scalar per pair); Hr = H gives every head its own landmarks.
 *   Head h uses retrieval head (Hr == 1 ? 0 : h).
 * - Retrieved sets are written in ascending chunk order, padded with index -1
 *   and score -inf.  Membership is decided by (score descending, chunk index
 *   ascending): ties go to the lower chunk index.
 * - Every element of every non-NULL output is written (zeros where the method
 *   gives nothing, e.g. the outputs of chunks 0 and 1 in CAUSAL mode).
 * - Arguments are validated before anything is launched; on error nothing is
 *   launched and a status != GCA_OK is returned, with detail in gca_last_error().
 *   Launch failures return GCA_ERR_HIP.  Kernel faults surface at the caller's
 *   next synchronisation.
 * - All work is enqueued on `stream`; no call synchronises (unless the
 *   environment variable GCA_DEBUG_SYNC is set to a value other than 0 when the
 *   library first launches: then every kernel launch is followed by a
 *   synchronisation of `stream` and an error check that names the kernel in
 *   gca_last_error(), for debugging).  Calls are
 *   re-entrant (no global mutable state besides the thread-local error string
 *   and the thread-local profiling hook below).
 * - Supported in this version: d == 64, S == 64, 1 <= topk <= 32, Hr in {1, H},
 *   D a positive multiple of 64 up to 8192, dtype FP32 or BF16 (all tensor
 *   inputs of a call share the dtype; scores, sel, w, lse, dsel and landmark
 *   gradients are always fp32).  Device pointers must be 16-byte aligned.
 */
#ifndef LIBGCA_GCA_H
#define LIBGCA_GCA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GCA_OK = 0,
  GCA_ERR_INVALID = 1,      /* malformed problem or NULL required pointer */
  GCA_ERR_UNSUPPORTED = 2,  /* well-formed but outside the supported shapes */
  GCA_ERR_WORKSPACE = 3,    /* workspace pointer NULL or smaller than required */
  GCA_ERR_HIP = 4           /* a HIP launch failed; see gca_last_error() */
} gca_status;

typedef enum { GCA_FP32 = 0, GCA_BF16 = 1 } gca_dtype;
typedef enum { GCA_CAUSAL = 0, GCA_DECODE = 1 } gca_mode;

/* Problem flags (gca_problem.flags). */
#define GCA_FLAG_FUSED_TOPK 1u   /* gca_forward, CAUSAL: score and select in one pass (no score matrix) */
#define GCA_FLAG_MATERIALIZE 2u  /* gca_forward, CAUSAL: always write the score matrix, then select */
#define GCA_FLAG_HOST_KV 8u      /* DECODE: k and v are pinned host allocations (hipHostMalloc),
                                  * the past chunks offloaded to CPU memory (Training &
                                  * Inference, "Memory Offloading"); landmarks, q and every
                                  * output stay in device memory.  The decode attention reads
                                  * the k retrieved chunks straight from host memory over the
                                  * host link (their device mapping, hipHostGetDevicePointer).
                                  * GCA_ERR_INVALID if k or v has no device mapping, or in
                                  * CAUSAL mode. */
#define GCA_FLAG_LMK_ROW 16u     /* CAUSAL: every query chunk has S + 1 rows, its S tokens followed
                                  * by its landmark (LMK) token (Methodology, Model Architecture:
                                  * the LMK token is inserted at the end of each chunk, and the
                                  * grouped cross attention of chunk t+1 takes its S + 1 hidden
                                  * states as queries against S-row retrieved chunks).  q, out,
                                  * lse, dout and dq then hold Lq = nQ * (S + 1) rows, row
                                  * c * (S + 1) + S being chunk c's LMK row; k, v, dk and dv keep
                                  * n_chunks * S rows.  The LMK row attends to and is fused over
                                  * the same retrieved set as its chunk's tokens.
                                  * GCA_ERR_UNSUPPORTED in DECODE mode. */
#define GCA_FLAG_GUMBEL 4u       /* Gumbel top-k selection (Training & Inference, "Gumbel Top-k
                                  * sampling"): every selection (gca_topk, gca_forward in both
                                  * modes) ranks score + g, g = -ln(-ln u) with u from the
                                  * Philox4x32-10 generator (Salmon et al., SC 2011) keyed by
                                  * gumbel_seed, counter (j / 4, t, b * Hr + hr, 0), word j mod 4,
                                  * u = (top 24 bits + 1/2) / 2^24 for candidate chunk j of
                                  * landmark row t (DECODE: t = 0).  sel, w and everything after
                                  * use the raw scores. */

/* Workspace queries (gca_workspace_size op argument). */
#define GCA_OP_FORWARD 0
#define GCA_OP_BACKWARD 1

/* The problem statement of Eq. 1-3: tokens per chunk S, top-k, heads H, head
 * dimension d, and the landmark representation width D. */
typedef struct {
  int32_t B;            /* batch */
  int32_t H;            /* attention heads */
  int32_t d;            /* head dimension (64) */
  int32_t S;            /* tokens per chunk (64) */
  int64_t n_chunks;     /* CAUSAL: chunks in the sequence; DECODE: past chunks */
  int32_t topk;         /* retrieved chunks per landmark row, 1..32 */
  int32_t Hr;           /* retrieval heads: 1 or H */
  int32_t D;            /* landmark vector width */
  float score_scale;    /* multiplies <landmark query, landmark key> (Eq. 1 uses 1/sqrt(D)) */
  float attn_scale;     /* multiplies <q, k> inside each chunk's attention (Eq. 3: 1/sqrt(d)) */
  int32_t off_by_one;   /* 0: plain softmax per chunk (Algorithm 1); 1: softmax-off-by-one (Eq. 3) */
  int32_t dtype;        /* gca_dtype of q, k, v, dout, dq, dk, dv, out, lmk_q, lmk_k */
  int32_t mode;         /* gca_mode */
  uint32_t flags;       /* GCA_FLAG_* */
  uint64_t gumbel_seed; /* generator seed for GCA_FLAG_GUMBEL (ignored otherwise) */
} gca_problem;

/* Causal relevance scores (Eq. 1):
 *   scores[b,hr,t,j] = score_scale * <lmk_q[b,hr,t,:], lmk_k[b,hr,j,:]>
 * for every j < t (CAUSAL) or every j (DECODE); -inf elsewhere.
 *   lmk_q  [B, Hr, nQ, D]        dtype      landmark queries (one per query chunk)
 *   lmk_k  [B, Hr, n_chunks, D]  dtype      landmark keys (one per chunk)
 *   scores [B, Hr, nQ, n_chunks] fp32       output
 */
gca_status gca_chunk_scores(const gca_problem* p, const void* lmk_q, const void* lmk_k,
                            float* scores, hipStream_t stream);

/* Top-k retrieval (Eq. 1): for each landmark row, the min(topk, #candidates)
 * best chunks, where candidates are the finite entries with j < t (CAUSAL) or
 * all finite entries (DECODE).
 *   scores [B, Hr, nQ, n_chunks] fp32   input (e.g. from gca_chunk_scores)
 *   idx    [B, Hr, nQ, topk]     int32  output: chunk indices ascending, -1 padded
 *   sel    [B, Hr, nQ, topk]     fp32   output: scores of the chosen chunks, -inf padded
 */
gca_status gca_topk(const gca_problem* p, const float* scores, int32_t* idx, float* sel,
                    hipStream_t stream);

/* Grouped cross attention forward (Eq. 2-3; Algorithm 1).  For every head h and
 * query chunk c with retrieval row t (CAUSAL: t = c-1; DECODE: t = 0) and every
 * valid slot s (idx >= 0) of that row:
 *   w[t,s]   = softmax over valid slots of sel[t,:]            (Eq. 2)
 *   P_s      = rowsoftmax(attn_scale * Q_c K_{j_s}^T)           (Eq. 3, per chunk)
 *   out_c    = sum_s w[t,s] * P_s V_{j_s}                       (Eq. 2)
 *   lse[., s]= log of slot s's softmax denominator (natural log, max included)
 * Rows whose retrieval row has no valid slot (CAUSAL chunks 0 and 1) get out = 0
 * and lse = -inf; pad slots get lse = -inf.  Slots with idx outside
 * [0, n_chunks) are treated as pads.
 *   q   [B, H, Lq, d]        dtype
 *   k,v [B, H, Lkv, d]       dtype
 *   idx [B, Hr, nQ, topk]    int32   (from gca_topk)
 *   sel [B, Hr, nQ, topk]    fp32    (from gca_topk; finite on valid slots)
 *   out [B, H, Lq, d]        dtype   output
 *   lse [B, H, Lq, topk]     fp32    output, may be NULL
 *   w   [B, Hr, nQ, topk]    fp32    output fusion weights, may be NULL
 */
gca_status gca_grouped_xattn_fwd(const gca_problem* p, const void* q, const void* k,
                                 const void* v, const int32_t* idx, const float* sel,
                                 void* out, float* lse, float* w, hipStream_t stream);

/* Backward of gca_grouped_xattn_fwd and of the score path (Algorithm 2, with the
 * gradient carried into the relevance scores through Eq. 2 and into the landmark
 * vectors through Eq. 1).  With dout the gradient of the loss w.r.t. out:
 *   dq, dk, dv [same shapes as q, k, v] dtype  gradients (dk/dv summed over every
 *                                             retrieval of each chunk)
 *   dsel   [B, Hr, nQ, topk] fp32  gradient w.r.t. the retrieved scores sel
 *                                  (0 on pad slots; the indices carry no gradient)
 *   dlmk_q [B, Hr, nQ, D]    fp32  gradient w.r.t. lmk_q (may be NULL)
 *   dlmk_k [B, Hr, n_chunks, D] fp32 gradient w.r.t. lmk_k (may be NULL)
 * lmk_q/lmk_k are needed only when dlmk_q/dlmk_k are requested (all four NULL
 * skips the landmark gradients; dlmk_q needs lmk_k, dlmk_k needs lmk_q).
 * lse must be the one written by gca_grouped_xattn_fwd for the same inputs.
 * The result is deterministic (no floating-point atomics).
 * Workspace: gca_workspace_size(p, GCA_OP_BACKWARD) bytes, 256-byte aligned.
 * GCA_ERR_UNSUPPORTED when nQ * topk exceeds INT32_MAX or nQ >= 2^26.
 */
gca_status gca_grouped_xattn_bwd(const gca_problem* p, const void* q, const void* k,
                                 const void* v, const int32_t* idx, const float* sel,
                                 const float* lse, const void* dout, void* dq, void* dk,
                                 void* dv, float* dsel, const void* lmk_q,
                                 const void* lmk_k, float* dlmk_q, float* dlmk_k,
                                 void* workspace, size_t ws_bytes, hipStream_t stream);

/* The whole forward path: scores (Eq. 1) -> top-k (Eq. 1) -> weights (Eq. 2) ->
 * grouped cross attention (Eq. 2-3).  Outputs as for the calls above; idx and sel
 * are required (the backward needs them), lse and w may be NULL.  In CAUSAL mode
 * the score matrix is written to the workspace and then selected, or, for long
 * sequences or with GCA_FLAG_FUSED_TOPK, scored and selected in one pass without
 * it.  In DECODE mode the past landmark keys are scanned in parallel ranges that
 * each leave their best k in the workspace; the attention kernel merges them
 * into idx/sel (the exact top-k) before attending.
 * Workspace: gca_workspace_size(p, GCA_OP_FORWARD) bytes, 256-byte aligned.
 */
gca_status gca_forward(const gca_problem* p, const void* lmk_q, const void* lmk_k,
                       const void* q, const void* k, const void* v, void* out,
                       int32_t* idx, float* sel, float* lse, float* w, void* workspace,
                       size_t ws_bytes, hipStream_t stream);

/* gca_forward for callers that cannot allocate memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * path and results as gca_forward on the same arguments, with the workspace
 * taken from a device array of GCA_NOALLOC_SCRATCH_BYTES that the library
 * holds on every device it runs on until the process ends.  The caller still
 * passes every input and output.  No memory is allocated or freed.
 * - GCA_ERR_UNSUPPORTED if gca_workspace_size(p, GCA_OP_FORWARD) exceeds
 *   GCA_NOALLOC_SCRATCH_BYTES (nothing is launched);
 * - all calls on one device share that device's array: calls that overlap in
 *   time on one device (different streams, or different threads without
 *   ordering) race on it and must not be issued.  Calls ordered on one stream
 *   are safe: no part of the array needs to start at any value, every byte a
 *   call reads was written earlier in the same call.
 * - GCA_ERR_HIP if the array's device address cannot be looked up (once per
 *   device, on the first call there). */
#define GCA_NOALLOC_SCRATCH_BYTES (16u << 20)
gca_status gca_forward_noalloc(const gca_problem* p, const void* lmk_q, const void* lmk_k,
                               const void* q, const void* k, const void* v, void* out,
                               int32_t* idx, float* sel, float* lse, float* w,
                               hipStream_t stream);

/* Profiling aid (outside the method).  While armed, the i-th kernel that libgca
 * launches from the calling thread (i = 0, 1, ... while 2 (i + 1) <= capacity,
 * capacity <= 4096) is dispatched with events[2 i] and events[2 i + 1] as its
 * start and stop events (hipExtLaunchKernel), so a caller can time each kernel
 * alone without adding work to the stream.  The events are created and owned
 * by the caller.  gca_profile_arm(NULL, 0) disarms; arming resets the count.
 * gca_profile_count() is the number of kernels timed since arming and
 * gca_profile_name(i) the name of kernel i (NULL if out of range). */
void gca_profile_arm(hipEvent_t* events, int capacity);
int gca_profile_count(void);
const char* gca_profile_name(int i);

/* Bytes of workspace `op` (GCA_OP_FORWARD or GCA_OP_BACKWARD) needs for problem p;
 * 0 if p is invalid or needs none. */
size_t gca_workspace_size(const gca_problem* p, int op);

/* Static description of a status code. */
const char* gca_status_string(gca_status s);

/* Detail of the last error raised on the calling thread ("" if none). */
const char* gca_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LIBGCA_GCA_H */
