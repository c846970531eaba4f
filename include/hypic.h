/*
 * hypic.h -- C ABI of libhypic.so, the MI355X (gfx950) hot path of
 * position-independent caching for gated-delta-rule (GDN) linear-attention
 * layers (Hypic, arXiv 2607.01299).
 *
 * Three operations:
 *   hypic_build_segment    zero-start prefill of independent segments, emitting
 *                          per-token outputs o, the zero-start end state S_{C|0}
 *                          and the segment-cumulative transition operator T_C
 *                          (Sec. 4.2 cache tuple; Sec. 5 state construction).
 *   hypic_compose_segments chains cached tuples behind a prefix state by the
 *                          composition law, Eq. (6).
 *   hypic_seam_rescan      runs the first w tokens of segments through the
 *                          recurrence from a composed incoming state, emitting
 *                          their outputs and the advanced state (Sec. 4.3, seam
 *                          propagation through linear-attention layers).
 * The same three for the scalar and diagonal transition families of Tab. 1
 * (hypic_family_build, hypic_family_compose, hypic_family_seam), and three
 * reuse-time steps next to the cache: the state RoPE shift of Eq. (7)
 * (hypic_rope_shift_state), the cached-key re-rotation of Eq. (8)
 * (hypic_rope_rerotate_keys) and the causal conv with a carried state
 * (hypic_causal_conv, Sec. 4.2 warm-up).  hypic_compose_with_seams reuses tail
 * tuples with seam windows that advance the state (Sec. 4.3).  hypic_kda_build
 * and hypic_kda_seam build and rescan the KDA row of Tab. 1 (delta rule with a
 * per-channel gate); its tuples compose with hypic_compose_segments.
 *
 * Math (Tab. 1 GDN row, Eq. (2)), per head, S in R^{d_k x d_v}:
 *   S_t = alpha_t (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T,
 *   o_t = S_t^T q_t          (the token reads the state after its own write),
 *   alpha_t = exp(log_alpha_t).
 * T_C is stored factored as in the Tab. 3 GDN closed form:
 *   T_C = exp(log_decay) * P_hat,  log_decay = sum_t log_alpha_t,
 *   P_hat = (I - beta_L k_L k_L^T) ... (I - beta_1 k_1 k_1^T)   (later tokens left).
 *
 * Conventions common to every entry point
 * ---------------------------------------
 * - Return value: HYPIC_OK (0) or a negative hypic_status.  Every argument is
 *   validated on the host before anything is enqueued; on error nothing is
 *   enqueued and no output is touched.
 * - Pointers are DEVICE pointers unless the name ends in _host (host memory,
 *   read only during the call).  The caller owns all memory; the library never
 *   allocates or frees device or host memory, keeps no pointer after
 *   returning and has no mutable global state, so calls are reentrant.
 * - Every call enqueues its kernels on `stream` (a hipStream_t; NULL means the
 *   default stream) and returns without synchronising.
 * - Layouts are dense row-major (C order).  Token tensors are packed:
 *     q, k : [T, h_qk, d_k]      v, o : [T, h_v, d_v]
 *     beta, log_alpha : [T, h_v] float32
 *   in the element type given by dims->dtype for q, k, v, o.  States, P_hat and
 *   log_decay are always float32.
 * - Grouped heads: h_v must be a multiple of h_qk; v-head h reads qk-head
 *   h / (h_v / h_qk).  beta and log_alpha are per v-head.
 * - Supported: d_k, d_v in {64, 128}; chunk in {16, 32, 64}; dtype F32 or BF16.
 *   Other values return HYPIC_EUNSUPPORTED.
 * - Device-side index arrays must hold the same values as their _host copies;
 *   the kernels clamp token ranges to [0, T) but do not re-validate.
 */
#ifndef HYPIC_H
#define HYPIC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hypic_status {
  HYPIC_OK = 0,
  HYPIC_EINVAL = -1,       /* bad pointer, size, offset or index */
  HYPIC_EUNSUPPORTED = -2, /* dims outside the supported set */
  HYPIC_EWORKSPACE = -3,   /* workspace missing or smaller than required */
  HYPIC_EHIP = -4          /* a HIP runtime call failed (launch error) */
} hypic_status;

typedef enum hypic_dtype { HYPIC_F32 = 0, HYPIC_BF16 = 1 } hypic_dtype;

typedef enum hypic_op {
  HYPIC_OP_BUILD = 0,
  HYPIC_OP_COMPOSE = 1,
  HYPIC_OP_SEAM = 2,
  HYPIC_OP_COMPOSE_RESCAN = 3
} hypic_op;

typedef struct hypic_dims {
  int32_t h_qk;  /* key/query heads */
  int32_t h_v;   /* value heads (multiple of h_qk) */
  int32_t d_k;   /* key dimension: 64 or 128 */
  int32_t d_v;   /* value dimension: 64 or 128 */
  int32_t dtype; /* hypic_dtype of q, k, v, o */
  int32_t chunk; /* tokens per chunk of the scan: 16, 32 or 64 */
} hypic_dims;

/* Bytes of device workspace `op` needs for `n` items (segments for BUILD,
 * requests for COMPOSE and COMPOSE_RESCAN, entries for SEAM).  Returns 0 when none is needed, and
 * 0 as well for invalid dims (the operation itself then reports the error). */
size_t hypic_workspace_bytes(int32_t op, const hypic_dims* dims, int64_t n);

/* Static, NUL-terminated description of a status code. */
const char* hypic_status_str(int32_t status);

/*
 * hypic_build_segment -- zero-start prefill of n_seg independent segments
 * (Sec. 4.2 cache tuple; Sec. 5: the end state from S_0 = 0 and the operator
 * from S_0 = I with writes zeroed; Tab. 3 GDN row for the factored operator).
 *
 *   q, k        [T, h_qk, d_k] dtype    v [T, h_v, d_v] dtype
 *   beta        [T, h_v] f32            log_alpha [T, h_v] f32 (any finite values)
 *   n_tokens    T, the rows of the packed token arrays (and of o).
 *   cu_seqlens  [n_seg + 1] int32 device; cu_seqlens_host the same values on the
 *               host: 0 = cu[0] <= cu[1] <= ... <= cu[n_seg] <= n_tokens, else
 *               HYPIC_EINVAL.  Segment s covers tokens [cu[s], cu[s+1]); a
 *               zero-length segment yields S_seg = 0, P_hat = I, log_decay = 0.
 *   o           [T, h_v, d_v] dtype, or NULL to skip the outputs.
 *   S_seg       [n_seg, h_v, d_k, d_v] f32: end state from S_0 = 0.
 *   P_hat       [n_seg, h_v, d_k, d_k] f32, or NULL to skip the operator path.
 *   log_decay   [n_seg, h_v] f32, or NULL.
 *   workspace   device scratch of at least
 *               hypic_workspace_bytes(HYPIC_OP_BUILD, dims, n_seg) bytes; that
 *               is 0 (workspace may be NULL) for n_seg <= 128, whose order
 *               travels in the kernel arguments.  Otherwise it holds the
 *               longest-first segment order, computed on the device;
 *               contents are not preserved across calls.
 * Segments are scheduled longest first (Eq. (9) LPT order, ties by index);
 * results do not depend on the schedule.  n_seg == 0 enqueues nothing.
 */
int32_t hypic_build_segment(const hypic_dims* dims, const void* q, const void* k,
                            const void* v, const float* beta,
                            const float* log_alpha, int32_t n_tokens,
                            const int32_t* cu_seqlens,
                            const int32_t* cu_seqlens_host, int32_t n_seg,
                            void* o, float* S_seg, float* P_hat,
                            float* log_decay, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * hypic_build_segment_noalloc -- hypic_build_segment for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  Same arguments and results as
 * hypic_build_segment without the workspace: the longest-first order of a
 * build of more than 128 segments goes into a fixed device array of the
 * library (one per GPU, HYPIC_NOALLOC_MAX_SEGMENTS int32 = 256 KiB, held until
 * the process ends) instead.  Allocates nothing and calls no allocating
 * routine.  n_seg > HYPIC_NOALLOC_MAX_SEGMENTS returns HYPIC_EWORKSPACE with
 * nothing enqueued.  `stream` must belong to the current device.  Every call on
 * a GPU shares that GPU's array: calls that overlap on one GPU (on different
 * streams, or concurrent host threads) race on it and must be serialised by
 * the caller; calls of up to 128 segments do not touch it.
 */
#define HYPIC_NOALLOC_MAX_SEGMENTS 65536
int32_t hypic_build_segment_noalloc(const hypic_dims* dims, const void* q, const void* k,
                                    const void* v, const float* beta,
                                    const float* log_alpha, int32_t n_tokens,
                                    const int32_t* cu_seqlens,
                                    const int32_t* cu_seqlens_host, int32_t n_seg,
                                    void* o, float* S_seg, float* P_hat,
                                    float* log_decay, void* stream);

/*
 * hypic_compose_segments -- Eq. (6): for each request r and v-head h, start
 * from S = S_prefix[r, h] (zero when S_prefix is NULL) and for each listed
 * segment i = seg_ids[j], j = req_offsets[r] .. req_offsets[r+1]-1 in order:
 *     S_incoming[j, h] = S;   S <- exp(log_decay[i, h]) * P_hat[i, h] @ S + S_seg[i, h]
 * then S_out[r, h] = S.
 *
 *   P_hat       [n_pool, h_v, d_k, d_k] f32   log_decay [n_pool, h_v] f32
 *   S_seg       [n_pool, h_v, d_k, d_v] f32   (the pool of cached tuples)
 *   seg_ids     [nnz] int32 device, seg_ids_host the same on the host, every
 *               value in [0, n_pool); nnz = req_offsets_host[n_req].
 *   req_offsets [n_req + 1] int32 device / req_offsets_host on the host:
 *               0 = off[0] <= off[1] <= ... (CSR).  A request with no segment
 *               returns its prefix.
 *   S_prefix    [n_req, h_v, d_k, d_v] f32 or NULL.
 *   S_out       [n_req, h_v, d_k, d_v] f32.
 *   S_incoming  [nnz, h_v, d_k, d_v] f32 or NULL.
 * P_hat, S_seg, S_prefix, S_out and S_incoming must be 16-byte aligned.
 * dims->dtype selects the arithmetic: F32 uses float32 matrix cores, BF16 uses
 * three-term split-bf16 products with float32 accumulation.  Workspace: none
 * (pass NULL, 0).  n_req == 0 enqueues nothing.
 */
int32_t hypic_compose_segments(const hypic_dims* dims, const float* P_hat,
                               const float* log_decay, const float* S_seg,
                               int32_t n_pool, const int32_t* seg_ids,
                               const int32_t* seg_ids_host,
                               const int32_t* req_offsets,
                               const int32_t* req_offsets_host, int32_t n_req,
                               const float* S_prefix, float* S_out,
                               float* S_incoming, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * hypic_seam_rescan -- Sec. 4.3 seam propagation through a linear-attention
 * layer: entry e covers tokens [tok_start[e], tok_start[e] + w_eff) of the packed
 * token arrays, w_eff = min(w, tok_len[e]); they run through the recurrence
 * starting from S_in[e] (the composed state entering the segment).
 *
 *   q, k, v, beta, log_alpha   packed token arrays as in build, n_tokens rows.
 *   tok_start, tok_len  [n_entries] int32 device; *_host the same on the host.
 *               Each tok_len >= 1 and tok_start + w_eff <= n_tokens.
 *   w           seam width, >= 1.
 *   S_in        [n_entries, h_v, d_k, d_v] f32.
 *   o_seam      [n_entries, w, h_v, d_v] dtype; rows >= w_eff are not written.
 *   S_post      [n_entries, h_v, d_k, d_v] f32 state after the w_eff tokens, or NULL.
 * Workspace: none (pass NULL, 0).  n_entries == 0 enqueues nothing.
 */
int32_t hypic_seam_rescan(const hypic_dims* dims, const void* q, const void* k,
                          const void* v, const float* beta,
                          const float* log_alpha, int32_t n_tokens,
                          const int32_t* tok_start, const int32_t* tok_len,
                          const int32_t* tok_start_host,
                          const int32_t* tok_len_host, int32_t n_entries,
                          int32_t w, const float* S_in, void* o_seam,
                          float* S_post, void* workspace,
                          size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Scalar and diagonal transition families (Tab. 1 rows without the delta-rule
 * correction; Tab. 3 compressed operators), through the same three steps.
 *
 * Per head and token t, with u_t = k_t v_t^T and Eq. (2):
 *   HYPIC_FAMILY_SCALAR   (RetNet, Lightning-2, Mamba2): S_t = exp(a_t) S_{t-1} + u_t
 *   HYPIC_FAMILY_DIAGONAL (GLA):             S_t = diag(exp(g_t)) S_{t-1} + u_t
 *   o_t = S_t^T q_t.
 * gate holds a_t as [T, h_v] float32 (scalar) or g_t as [T, h_v, d_k] float32
 * (diagonal), natural-log units.  The segment operator T_C of Tab. 3 is a
 * scalar exp(sum_t a_t) or a vector exp(sum_t g_t); it is returned as its
 * logarithm log_decay, [n, h_v] (scalar) or [n, h_v, d_k] (diagonal), which
 * does not underflow on long segments.
 *
 * The diagonal family's chunked kernel refers each key's gate to the start of
 * its 16-token tile, so every channel's gate sum over any 16 consecutive tokens
 * must be above -80 (float32 range; e.g. per-token gates >= -5); beyond that the
 * outputs are undefined.  The scalar family has no such limit.
 * dims->chunk is validated but the family kernels always run chunks of 64
 * tokens (results do not depend on the chunk size).  Other conventions as above.
 * ------------------------------------------------------------------------ */
typedef enum hypic_family {
  HYPIC_FAMILY_SCALAR = 1,
  HYPIC_FAMILY_DIAGONAL = 2
} hypic_family;

/*
 * hypic_family_build -- zero-start prefill of n_seg independent segments of a
 * scalar- or diagonal-family layer (Sec. 4.2 cache tuple, Tab. 3 compressed
 * operator).
 *   q, k [T, h_qk, d_k] dtype; v [T, h_v, d_v] dtype; gate as above.
 *   n_tokens, cu_seqlens / cu_seqlens_host, o, S_seg, workspace: as in
 *   hypic_build_segment.
 *   log_decay   [n_seg, h_v] (scalar) or [n_seg, h_v, d_k] (diagonal) f32, or NULL.
 * A zero-length segment yields S_seg = 0 and log_decay = 0.
 * Returns HYPIC_EUNSUPPORTED for an unknown family.
 */
int32_t hypic_family_build(const hypic_dims* dims, int32_t family, const void* q,
                           const void* k, const void* v, const float* gate, int32_t n_tokens,
                           const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                           int32_t n_seg, void* o, float* S_seg, float* log_decay,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * hypic_family_compose -- Eq. (6) with the compressed operators of Tab. 3: for
 * each request r and v-head h, S = S_prefix[r, h] (zero when NULL); for each
 * listed segment i = seg_ids[j] in order
 *     S_incoming[j, h] = S;   S <- exp(log_decay[i, h]) . S + S_seg[i, h]
 * (scalar: one factor; diagonal: row c of S scaled by exp(log_decay[i, h, c]));
 * then S_out[r, h] = S.  Arguments as in hypic_compose_segments, without P_hat;
 * S_seg, S_prefix, S_out and S_incoming must be 16-byte aligned.  The
 * arithmetic is float32 whatever dims->dtype says.  Workspace: none.
 */
int32_t hypic_family_compose(const hypic_dims* dims, int32_t family, const float* log_decay,
                             const float* S_seg, int32_t n_pool, const int32_t* seg_ids,
                             const int32_t* seg_ids_host, const int32_t* req_offsets,
                             const int32_t* req_offsets_host, int32_t n_req,
                             const float* S_prefix, float* S_out, float* S_incoming,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * hypic_family_seam -- Sec. 4.3 seam rescan for a scalar- or diagonal-family
 * layer: entry e runs tokens [tok_start[e], tok_start[e] + min(w, tok_len[e]))
 * through the family's recurrence from S_in[e].  Arguments and outputs as in
 * hypic_seam_rescan with gate in place of beta and log_alpha (w may exceed 64).
 * Workspace: none.
 */
int32_t hypic_family_seam(const hypic_dims* dims, int32_t family, const void* q, const void* k,
                          const void* v, const float* gate, int32_t n_tokens,
                          const int32_t* tok_start, const int32_t* tok_len,
                          const int32_t* tok_start_host, const int32_t* tok_len_host,
                          int32_t n_entries, int32_t w, const float* S_in, void* o_seam,
                          float* S_post, void* workspace, size_t workspace_bytes,
                          void* stream);

/*
 * hypic_kda_build -- Sec. 4.2 cache tuples for a layer of the KDA row of Tab. 1:
 *     S_t = (I - beta_t k_t k_t^T) diag(exp(g_t)) S_{t-1} + beta_t k_t v_t^T,
 *     o_t = S_t^T q_t,
 * from S = 0 for every segment, with the Tab. 3 operator
 *     T_C = prod_t (I - beta_t k_t k_t^T) diag(exp(g_t))   (later tokens left)
 * stored as T_C = exp(log_decay) * P_hat.  log_decay is the sum, over the
 * segment's chunks of 64 tokens from its start, of each chunk's largest
 * per-channel gate sum (a scale that keeps P_hat in float32 range); the tuple
 * (P_hat, log_decay, S_seg) composes with hypic_compose_segments unchanged.
 *   q, k, v, beta, n_tokens, cu_seqlens, o, S_seg  as in hypic_build_segment.
 *   gate      [T, h_v, d_k] float32: the per-channel log gates g_t (natural log).
 *   P_hat     [n_seg, h_v, d_k, d_k] float32 or NULL (no operator; then
 *             log_decay is not written).
 *   log_decay [n_seg, h_v] float32, written with P_hat.
 * q, k, v 16-byte aligned.  The chunked kernel refers each key's gate to its
 * 16-token tile: every channel's gate sum over any 16 consecutive tokens of a
 * segment must stay above about -80, else results lose float32 range.
 * Workspace: hypic_workspace_bytes(HYPIC_OP_BUILD, dims, n_seg) bytes (the
 * longest-first order of more than 128 segments), as for the GDN build.
 */
int32_t hypic_kda_build(const hypic_dims* dims, const void* q, const void* k, const void* v,
                        const float* beta, const float* gate, int32_t n_tokens,
                        const int32_t* cu_seqlens, const int32_t* cu_seqlens_host, int32_t n_seg, void* o, float* S_seg,
                        float* P_hat, float* log_decay, void* workspace, size_t workspace_bytes,
                        void* stream);

/*
 * hypic_kda_seam -- Sec. 4.3 seam rescan for a KDA layer: entry e runs tokens
 * [tok_start[e], tok_start[e] + min(w, tok_len[e])) through the KDA recurrence
 * from S_in[e].  Arguments and outputs as in hypic_seam_rescan with the
 * per-channel gate [n_tokens, h_v, d_k] in place of log_alpha (w may exceed 64).
 * Workspace: none.
 */
int32_t hypic_kda_seam(const hypic_dims* dims, const void* q, const void* k, const void* v,
                       const float* beta, const float* gate, int32_t n_tokens,
                       const int32_t* tok_start, const int32_t* tok_len,
                       const int32_t* tok_start_host, const int32_t* tok_len_host,
                       int32_t n_entries, int32_t w, const float* S_in, void* o_seam,
                       float* S_post, void* workspace, size_t workspace_bytes, void* stream);

/*
 * hypic_compose_with_seams -- reuse with seam windows that advance the state
 * (Sec. 4.3: the first w tokens of each reused segment are left out of its
 * cached tuple and recomputed through the layer from the composed state).
 * Pool entry i is cached as the tuple of its tail, the tokens
 * [seam_start[i] + w_i, seam_start[i] + seam_len[i]) with w_i = min(w, seam_len[i])
 * (built with hypic_build_segment over those tokens), and its seam is its first
 * w_i tokens.  For each request r and v-head h, from S = S_prefix[r, h] (zero
 * when NULL), each listed entry i = seg_ids[j] in order does
 *     (o_seam[j, 0 .. w_i - 1, h], S) = the recurrence of Eq. (2) over the seam from S;
 *     S <- exp(log_decay[i, h]) * P_hat[i, h] @ S + S_seg[i, h]        (Eq. (4))
 * then S_out[r, h] = S.  Composing the tail tuples this way equals the
 * recurrence over the concatenated segments.
 *   P_hat, log_decay, S_seg  the pool of tail tuples, as in hypic_compose_segments.
 *   q, k, v, beta, log_alpha  packed token arrays ([n_tokens, ...], as in the build)
 *                            holding every entry's seam tokens.
 *   seam_start, seam_len [n_pool] int32 device / _host: first token and segment
 *                            length of entry i (seam_len >= 1; seam_start + w_i <= n_tokens).
 *   w                        seam width >= 1.
 *   seg_ids, req_offsets     CSR request lists as in hypic_compose_segments.
 *   S_prefix [n_req, h_v, d_k, d_v] f32 or NULL; S_out [n_req, h_v, d_k, d_v] f32
 *                            (16-byte aligned).
 *   o_seam [nnz, w, h_v, d_v] dtype, in the CSR order of seg_ids; rows >= w_i
 *                            are not written.
 *   workspace  at least hypic_seam_compose_workspace_bytes(dims, n_req, max_n)
 *              bytes, max_n = the longest request's entry count: two running
 *              states per request and the per-step entry lists.
 * dims->dtype gives the token type and the composition arithmetic as in
 * hypic_seam_rescan and hypic_compose_segments.  Requests run longest first
 * (Eq. (9) list order).  With bf16 tokens, chunk 64 and w <= 64 the call is one
 * launch in which each (request, head) keeps its running state on chip across
 * its entries (seam, then Eq. (4) with the entry's tail tuple); otherwise each
 * step enqueues one seam and one composition launch over the requests still
 * running.
 */
size_t hypic_seam_compose_workspace_bytes(const hypic_dims* dims, int32_t n_req,
                                          int32_t max_per_request);
int32_t hypic_compose_with_seams(const hypic_dims* dims, const float* P_hat,
                                 const float* log_decay, const float* S_seg, int32_t n_pool,
                                 const void* q, const void* k, const void* v, const float* beta,
                                 const float* log_alpha, int32_t n_tokens,
                                 const int32_t* seam_start, const int32_t* seam_start_host,
                                 const int32_t* seam_len, const int32_t* seam_len_host, int32_t w,
                                 const int32_t* seg_ids, const int32_t* seg_ids_host,
                                 const int32_t* req_offsets, const int32_t* req_offsets_host,
                                 int32_t n_req, const float* S_prefix, float* S_out,
                                 void* o_seam, void* workspace, size_t workspace_bytes,
                                 void* stream);

/*
 * hypic_compose_and_rescan -- Eq. (6) composition with each listed segment's
 * seam window rescanned from the state entering it, in one pass (Sec. 4.3;
 * the cached tuples cover whole segments and the seam does not advance the
 * composed state).  For each request r and v-head h, from S = S_prefix[r, h]
 * (zero when NULL), each listed entry i = seg_ids[j] in order does
 *     o_seam[j, 0 .. w_i - 1, h] = outputs of the recurrence of Eq. (2) over
 *                                  the entry's first w_i tokens from S;
 *     S <- exp(log_decay[i, h]) * P_hat[i, h] @ S + S_seg[i, h]        (Eq. (4))
 * then S_out[r, h] = S: the results of hypic_compose_segments (S_out) and of
 * hypic_seam_rescan on its incoming states (o_seam), without writing or
 * reading the incoming states.  Each (request, head) keeps its state on chip.
 *   Arguments as in hypic_compose_with_seams, except that the pool holds
 *   whole-segment tuples and seam_start / seam_len give each pool entry's
 *   first token and length (w_i = min(w, seam_len[i])).
 *   Requires bf16 tokens (dims->dtype == HYPIC_BF16, split-bf16 composition),
 *   chunk 64 and w <= 64, else HYPIC_EUNSUPPORTED.
 *   workspace  hypic_workspace_bytes(HYPIC_OP_COMPOSE_RESCAN, dims, n_req) bytes:
 *              0 up to 128 requests (their longest-first order travels in the
 *              kernel arguments), else the order, computed on the device.
 */
int32_t hypic_compose_and_rescan(const hypic_dims* dims, const float* P_hat,
                                 const float* log_decay, const float* S_seg, int32_t n_pool,
                                 const void* q, const void* k, const void* v, const float* beta,
                                 const float* log_alpha, int32_t n_tokens,
                                 const int32_t* seam_start, const int32_t* seam_start_host,
                                 const int32_t* seam_len, const int32_t* seam_len_host, int32_t w,
                                 const int32_t* seg_ids, const int32_t* seg_ids_host,
                                 const int32_t* req_offsets, const int32_t* req_offsets_host,
                                 int32_t n_req, const float* S_prefix, float* S_out,
                                 void* o_seam, void* workspace, size_t workspace_bytes,
                                 void* stream);

/* ------------------------------------------------------------------------
 * Reuse-time steps next to the linear-attention cache.
 * R(p) is the rotary position embedding: it rotates channel pairs (2i, 2i+1)
 * of a d-vector by p * base^(-2i/d).  Angles are formed in float64.
 * ------------------------------------------------------------------------ */

/*
 * hypic_rope_shift_state -- Eq. (7): a state cached with its keys rotated for
 * positions starting at a is moved to positions starting at b by rotating its
 * d_k rows, S_out[e, h] = R(delta[e]) S_in[e, h] with delta[e] = b - a.  Exact
 * for transitions that commute with R (the scalar family; pair-shared gates).
 *   S_in, S_out  [n, h_v, d_k, d_v] f32, 16-byte aligned; S_out may equal S_in.
 *   delta        [n] int32 device.
 *   base         RoPE base (> 0, finite).
 */
int32_t hypic_rope_shift_state(const hypic_dims* dims, const float* S_in, float* S_out,
                               int32_t n, const int32_t* delta, double base, void* stream);

/*
 * hypic_rope_rerotate_keys -- Eq. (8): cached keys of segment s rotated from
 * positions starting at a to positions starting at b, k_out = R(delta[s]) k_in
 * for each of its tokens and heads, delta[s] = b - a (values are unchanged).
 *   k_in, k_out  [T, h_qk, d_k] in dims->dtype, 16-byte aligned; k_out may equal k_in.
 *   cu_seqlens   [n_seg + 1] int32 device / _host as in hypic_build_segment;
 *                the longest segment must be under 4,194,240 tokens.
 *   delta        [n_seg] int32 device.
 */
int32_t hypic_rope_rerotate_keys(const hypic_dims* dims, const void* k_in, void* k_out,
                                 const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                                 int32_t n_seg, const int32_t* delta, double base,
                                 void* stream);

/*
 * hypic_causal_conv -- the depthwise causal convolution in front of a
 * linear-attention layer, over packed segments with a carried conv state
 * (Sec. 4.2: a segment cached on its own starts from zeros; at reuse its
 * first width - 1 outputs are recomputed from the previous segment's state):
 *   y[t, c] = act(sum_{j < width} weight[c, j] * xx[t + j, c]),
 *   xx = concat(state_in[s], x[tokens of segment s]),  act = SiLU if silu else identity,
 *   state_out[s] = the last width - 1 rows of xx.
 *   x, y        [T, channels] in dtype (HYPIC_F32 or HYPIC_BF16), 16-byte aligned;
 *               y must not alias x.
 *   weight      [channels, width] f32, 1 <= width <= 8.
 *   state_in    [n_seg, width - 1, channels] f32, or NULL for zeros.
 *   state_out   [n_seg, width - 1, channels] f32, or NULL.
 */
int32_t hypic_causal_conv(int32_t dtype, int32_t channels, int32_t width, const void* x,
                          const float* weight, const int32_t* cu_seqlens,
                          const int32_t* cu_seqlens_host, int32_t n_seg, const float* state_in,
                          void* y, float* state_out, int32_t silu, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HYPIC_H */
