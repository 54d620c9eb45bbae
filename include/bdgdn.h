/*
 * bdgdn.h -- C ABI of the block-diffusion Gated DeltaNet library (libbdgdn.so) for
 * AMD MI355X (gfx950).
 *
 * The library computes the Gated Delta Rule (GDR) layer of FLARE's hybrid backbone
 * (arXiv 2606.01774) under the block-diffusion clean/noisy schedule:
 *
 *   clean stream (Sec. 3.1, eq. gdn-recurrence; Appendix eq. per-step-fwd):
 *     S_t = exp(g_t) (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T,
 *     o_t = scale * S_t^T q_t                                (S is d_k x d_v)
 *   noisy stream (Sec. 3.2, eq. flare-gdn-schedule; Appendix eq. noisy-block-fwd):
 *     block b of L positions is seeded with the clean state after the last clean
 *     position before the block, applies its own L noisy updates, and every
 *     position of the block reads the block-end noisy state:
 *     on_l = scale * Sn_end^T qn_l.
 *   document packing (Appendix "Document-packed training"): documents start on
 *     block boundaries, each starts from a zero state, the last block of a document
 *     may be partial (treated as padded with identity positions).
 *   serving (Appendix "Diffusion-Trust Sampling", "Differences between the denoise
 *     pass and the state-update pass"): a denoise pass reads the cached state and
 *     never writes it; a commit pass runs the token-causal update and writes it back.
 *
 * Conventions shared by every entry point
 *   - Pointers named *_dev / tensors are device pointers (HIP device memory); the
 *     only host pointers are the descriptors and cu_seqlens_host.
 *   - Token tensors are token-major and contiguous:
 *       q, k : [rows][h_qk][d_k]      v, o : [rows][h_v][d_v]     g, beta : [rows][h_v]
 *     where rows = batch*seqlen (training) or num_req*block (serving).
 *     q, k, v have the descriptor's dtype and o its out_dtype; g (the LOG gate,
 *     alpha = exp(g)) and beta are fp32 and used as given.  g must be <= 0 (alpha in
 *     (0, 1], a decay): the bf16 kernels evaluate every decay exponent as non-positive,
 *     and a positive g gives unspecified (finite) results there.
 *   - Arithmetic: states and all accumulations are fp32.  With bf16 inputs the MFMA
 *     operands are fp16 (the bf16 values converted exactly; every rounded
 *     intermediate keeps 11 significant bits), so inputs and intermediates must stay
 *     within fp16 range: |q|, |k|, |v| and state entries below 2^15 (q and k are
 *     normally L2-normalised); magnitudes below 2^-14 lose relative precision
 *     (absolute error under 2^-25).  With fp32 inputs everything is fp32.
 *   - v-head h reads q/k head h / (h_v / h_qk) (consecutive grouping).
 *   - States are fp32 [unit][h_v][d_k][d_v], row-major (paper orientation).
 *   - All work is enqueued on `stream` (a hipStream_t; NULL = default stream); no
 *     call synchronises the host or allocates device memory.  Outputs are valid
 *     once the stream reaches that point.
 *   - Every argument is validated on the host before anything is launched.  On
 *     any error return nothing is launched and no output is touched.
 *   - q, k, v and the dtype outputs must be 16-byte aligned (BDGDN_ERR_INVALID_ARG).
 *   - The caller owns every buffer.  Outputs must not alias inputs.
 *   - Calls are thread-safe; the library keeps no mutable global state besides a
 *     once-initialised table of kernel attributes.
 *
 * Supported: d_k, d_v in {64, 128}; 1 <= block <= 64; (dtype, out_dtype) in
 * {(bf16, fp32), (bf16, bf16), (fp32, fp32)}, fp32 inputs with block <= 32.
 * Anything else returns BDGDN_ERR_UNSUPPORTED.  fp32 outputs for bf16 inputs are the
 * accuracy-grade choice: rounding an output to bf16 alone perturbs it by up to
 * 2^-9 of its magnitude.
 */
#ifndef BDGDN_H
#define BDGDN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BDGDN_OK               0
#define BDGDN_ERR_INVALID_ARG -1 /* NULL required pointer, non-positive size, h_v % h_qk != 0,
                                    non-finite scale, inconsistent cu_seqlens */
#define BDGDN_ERR_UNSUPPORTED -2 /* (dtype, d_k, d_v, block) outside the supported set */
#define BDGDN_ERR_UNALIGNED   -3 /* a document start cu_seqlens[i] (i < N) is not a multiple
                                    of block (Appendix "Document-packed training") */
#define BDGDN_ERR_WORKSPACE   -4 /* workspace smaller than bdgdn_fwd_train_workspace() */
#define BDGDN_ERR_LAUNCH      -5 /* the HIP runtime reported an error for a launch */
#define BDGDN_ERR_SCRATCH     -6 /* the input needs more than the fixed scratch of a
                                    no-allocation entry point (nothing is launched) */

typedef enum { BDGDN_BF16 = 0, BDGDN_F32 = 1 } bdgdn_dtype_t;

/* How the training forward is scheduled; every route gives the same result up to
 * floating-point summation order.
 *  FUSED:   the fused two-stream schedule (Appendix "Route II"): one workgroup per
 *           (sequence, v-head, d_v tile) scans the blocks in order with the clean state
 *           on chip and evaluates each noisy block from the in-register boundary state.
 *           With bf16 inputs and blocks of at most 32 positions this is one kernel whose
 *           workgroups also compute each block's UT transform and masked Q K^T a block
 *           ahead (no workspace); when (sequences or documents) x v-heads reach the
 *           GPU's 256 compute units and d_k = d_v, one workgroup per (sequence, v-head)
 *           covers all d_v columns instead (CHUNKED's output pass with one segment per
 *           chain; no workspace).  Blocks of an even 34 .. 64 positions run the one
 *           kernel on sub-blocks of half the block, each noisy block carrying its state
 *           across its two halves (no workspace).  Blocks of 1, 2, 4 or 8 positions run
 *           it on 32-position clean chunks that hold 32 / block noisy blocks each, every
 *           noisy block seeded on chip with the clean state at its own start (no
 *           workspace).  Otherwise it is the RECORDS schedule.
 *  SPLIT:   boundary states through HBM and a separate noisy-block kernel (Appendix
 *           "Route I"): the clean scan writes the clean state before every block (the
 *           seed of that noisy block) into the workspace, fp32 [block][h_v][d_k][d_v]
 *           (blocks of all sequences, or of the packed axis, in order), then every
 *           noisy block is evaluated in parallel from its seed.  The clean outputs and
 *           ht equal FUSED's bit for bit.  bf16 inputs, d_k = d_v = 128 and blocks of at
 *           most 32 positions only (else BDGDN_ERR_UNSUPPORTED).
 *  ONEPASS: one kernel per (sequence, v-head, d_v tile) that recomputes the UT
 *           transform of each block itself, without overlap.  No workspace.
 *  RECORDS: two kernels: the UT transform and masked Q K^T of every (block, v-head)
 *           in parallel into the workspace, then the scan of FUSED reading them.
 *           Needs a workspace (bdgdn_fwd_train_workspace).
 *  CHUNKED: the chunk-parallel schedule (Appendix "Route II" with the chunk-state pass
 *           of eq. chunk-state): every (sequence or document, v-head) chain is cut into
 *           segments of G blocks, G a power of two >= 16 chosen from the descriptor so
 *           that the (chain, segment) pairs cover the GPU's compute units; a state pass
 *           computes the clean state at every later segment start (with the blocks'
 *           clean UT transforms computed in parallel before it), then one workgroup per
 *           (chain, segment) evaluates the segment's blocks for all d_v columns at once.
 *           Needs a workspace (bdgdn_fwd_train_workspace): a clean UT record per
 *           (block, v-head) and an fp32 state per (later segment start, v-head).  bf16
 *           inputs, d_k = d_v in {64, 128}, blocks of at most 32 positions, at most 512
 *           packed documents (else BDGDN_ERR_UNSUPPORTED). */
typedef enum {
    BDGDN_ROUTE_FUSED = 0,
    BDGDN_ROUTE_SPLIT = 1,
    BDGDN_ROUTE_ONEPASS = 2,
    BDGDN_ROUTE_RECORDS = 3,
    BDGDN_ROUTE_CHUNKED = 4
} bdgdn_route_t;

typedef struct {
    int32_t batch;     /* B sequences; must be 1 when packed (num_seqs > 0)            */
    int32_t seqlen;    /* T tokens per sequence, or total packed tokens                 */
    int32_t num_seqs;  /* N packed documents, 0 when not packed                         */
    int32_t h_qk, h_v; /* q/k heads and v heads; h_v % h_qk == 0                        */
    int32_t d_k, d_v;  /* head dimensions                                               */
    int32_t block;     /* diffusion block size L                                        */
    float scale;       /* output scale s (the paper uses 1/sqrt(d_k))                   */
    int32_t dtype;     /* bdgdn_dtype_t of q, k, v                                      */
    int32_t route;     /* bdgdn_route_t                                                 */
    int32_t out_dtype; /* bdgdn_dtype_t of o, on                                        */
} bdgdn_fwd_desc_t;

typedef struct {
    int32_t num_req;   /* R requests, one block of `block` tokens each                  */
    int32_t h_qk, h_v, d_k, d_v;
    int32_t block;     /* L                                                             */
    float scale;
    int32_t dtype;     /* bdgdn_dtype_t of q, k, v                                      */
    int32_t out_dtype; /* bdgdn_dtype_t of o / o_causal                                 */
} bdgdn_serve_desc_t;

/* Library version, (major << 16) | minor. */
int32_t bdgdn_version(void);

/* Human-readable text of a status code (static storage). */
const char *bdgdn_status_string(int status);

/* Bytes of device workspace bdgdn_fwd_train needs for this descriptor (0 when the
 * route runs without one), or 0 for a descriptor that bdgdn_fwd_train would reject. */
size_t bdgdn_fwd_train_workspace(const bdgdn_fwd_desc_t *desc);

/*
 * Two-stream training forward (clean + noisy), Sec. 3.2 and Appendix "Gated Delta
 * Rule: two-stream training".
 *
 *   q, k, v, g, beta       clean stream   ([B*T] rows, layouts above)
 *   qn, kn, vn, gn, betan  noisy stream   (same shapes; gn/betan are the noisy
 *                                          stream's own gates)
 *   cu_seqlens_dev/_host   both NULL (B sequences of T tokens) or both [N+1] int32
 *                          offsets into the packed axis (B == 1, cu[0] == 0,
 *                          cu[N] == T, non-decreasing, cu[i] % block == 0 for i < N).
 *                          The two copies must hold the same values.
 *   h0                     [B or N][h_v][d_k][d_v] fp32 initial clean state, or NULL
 *                          for zero.  Each sequence's first noisy block is seeded
 *                          with the same state.
 *   o, on                  [B*T][h_v][d_v] outputs of out_dtype (clean causal readout,
 *                          noisy block-end readout); every row is written.
 *   ht                     [B or N][h_v][d_k][d_v] fp32 final clean state, or NULL.
 *   workspace              device memory of at least bdgdn_fwd_train_workspace(desc)
 *                          bytes, 256-byte aligned (may be NULL when that is 0); its
 *                          contents are scratch owned by the call until the stream
 *                          passes it.
 * Returns BDGDN_OK or a negative status.
 */
int bdgdn_fwd_train(const bdgdn_fwd_desc_t *desc,
                    const void *q, const void *k, const void *v,
                    const float *g, const float *beta,
                    const void *qn, const void *kn, const void *vn,
                    const float *gn, const float *betan,
                    const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                    const float *h0, void *o, void *on, float *ht,
                    void *workspace, size_t workspace_bytes, void *stream);

/*
 * Complementary-view training forward (Sec. 3.3 "Training Objective and Mask Design": each
 * block is trained under two complementary noisy views, both conditioned on the same clean
 * context): one clean scan, whose boundary states seed every block of every noisy view.
 * Each view is a noisy stream of its own (inputs, gates, block-end readout); view i's output
 * equals the `on` of bdgdn_fwd_train with the same clean stream and view i as the noisy
 * stream.  desc->route picks the schedule:
 *   FUSED  one pass of the one-kernel forward per view, the clean scan recomputed with each
 *          view and every noisy block evaluated from the on-chip boundary state (no
 *          workspace);
 *   SPLIT  one pass of the one-kernel forward over the clean stream and view 0 that also
 *          writes the seed state of every (block, v-head) to the workspace, then the
 *          noisy-block pass from the seeds for every further view (the clean scan runs once;
 *          the seeds make a round trip through device memory).
 * Other routes give BDGDN_ERR_UNSUPPORTED.
 */
typedef struct {
    const void *q, *k, *v;   /* [B*T][h_qk or h_v][d] of desc->dtype, 16-byte aligned */
    const float *g, *beta;   /* [B*T][h_v] fp32: the view's log-gates and step sizes  */
    void *o;                 /* [B*T][h_v][d_v] of desc->out_dtype: its readout       */
} bdgdn_noisy_view_t;

/* Bytes of workspace bdgdn_fwd_train_views needs: the seed states for the SPLIT route, 0
 * for FUSED or for a descriptor it would reject. */
size_t bdgdn_fwd_train_views_workspace(const bdgdn_fwd_desc_t *desc);

/* Clean inputs, h0, o, ht and cu_seqlens as for bdgdn_fwd_train; views[0 .. n_views-1],
 * 1 <= n_views <= 16.  bf16 inputs; FUSED takes the blocks the one-kernel forward takes (at
 * most 32 positions, or an even 34 .. 64), SPLIT needs d_k = d_v = 128 and blocks of at most
 * 32 positions (else BDGDN_ERR_UNSUPPORTED). */
int bdgdn_fwd_train_views(const bdgdn_fwd_desc_t *desc,
                          const void *q, const void *k, const void *v,
                          const float *g, const float *beta,
                          const bdgdn_noisy_view_t *views, int32_t n_views,
                          const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                          const float *h0, void *o, float *ht,
                          void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of device workspace bdgdn_bwd_train needs.  Block-form shapes (bf16 inputs,
 * d_k = d_v = 128, blocks of at most 32 positions), per (block, v-head): the recomputed
 * clean seed state (fp16), the part of the clean state gradient at the block's start that
 * does not depend on the gradient at its end (fp16; overwritten by the gradient at the
 * block's end once the reverse scan has read it), the block's U K (32 x d_k fp16) and
 * gamma_n; plus 2.3 KB for the range pass.  Per-step shapes: the clean state before every
 * eighth block of every chain (fp32) and eight block-start states per (chain, 16-column
 * tile) (fp32).  0 for a descriptor it would reject. */
size_t bdgdn_bwd_train_workspace(const bdgdn_fwd_desc_t *desc);

/* Bytes of device workspace bdgdn_bwd_train (and bdgdn_bwd_train_views) needs when run in
 * `segments` time segments (Appendix "Backward primitives": the strided clean-state
 * checkpoints of the checkpoint build, with the stride chosen as in "Choosing the stride"):
 * every chain's clean blocks (sub-blocks of half the block for blocks of 34 .. 64) are cut
 * into segments of ceil(longest chain's blocks / segments) (even for sub-blocks), the clean
 * state at each segment start after the first is kept (fp32, one per (sequence, v-head)),
 * and the segments run last first, each recomputing its own seeds from its checkpoint, so
 * that the per-block workspace above holds the first segment's blocks only (for every
 * sequence, min(its blocks, the segment length)), plus the checkpoints, one fp32
 * state-gradient carry per (sequence, v-head) and the segment tables.
 *   cu_seqlens_host   [N+1] document offsets when desc->num_seqs > 0, else NULL
 *   segments          >= 1; 1 gives bdgdn_bwd_train_workspace(desc); more than the longest
 *                     chain's blocks count as that many
 * Per-step shapes need no more than bdgdn_bwd_train_workspace(desc) and are never segmented
 * (that value for any segments).  0 for a descriptor it would reject or missing packing. */
size_t bdgdn_bwd_train_workspace_segmented(const bdgdn_fwd_desc_t *desc, const int32_t *cu_seqlens_host,
                                           int segments);

/*
 * Backward of bdgdn_fwd_train (Appendix "Backward primitives": the noisy block-end
 * readout backward, eq. noisy-readout-bwd; the block-level chain rule,
 * eq. dh-block-recursion; the clean chunk backward): the gradients of
 *     sum <do, o> + sum <don, on> + <dht, ht>
 * with respect to every input of the forward, for the same descriptor and inputs
 * (desc->route is not used; desc->out_dtype is the dtype of do and don).
 *
 *   do, don              [B*T][h_v][d_v] upstream gradients of o and on (out_dtype)
 *   dht                  [B or N][h_v][d_k][d_v] fp32 gradient of ht, or NULL for zero
 *   dq, dk, dqn, dkn     [B*T][h_qk][d_k] fp32 (summed over the v-heads of a q/k head)
 *   dv, dvn              [B*T][h_v][d_v] fp32
 *   dg, dbeta, dgn, dbetan  [B*T][h_v] fp32 (gradients of the log-gates and step sizes)
 *   dh0                  [B or N][h_v][d_k][d_v] fp32 gradient of h0, or NULL
 *   workspace            256-byte aligned, owned by the call until the stream passes it;
 *                        at least bdgdn_bwd_train_workspace(desc) bytes runs the blocks of
 *                        every chain at once.  A smaller one runs the block-form shapes in
 *                        the fewest time segments s >= 2 with
 *                        bdgdn_bwd_train_workspace_segmented(desc, cu_seqlens_host, s) <=
 *                        workspace_bytes (the same results bit for bit: the checkpoints
 *                        and the carry are the fp32 values the one-pass call keeps on
 *                        chip; one more clean-scan pass over all but the last segment and
 *                        more, smaller launches); BDGDN_ERR_WORKSPACE if none fits
 * Every gradient row is overwritten.  bf16 inputs with d_k = d_v = 128 and blocks of at
 * most 32 positions run the block-form kernels; fp32 inputs (blocks of at most 32), d_k or
 * d_v of 64, and bf16 blocks of 33 .. 64 positions run the per-step fp32 backward (one
 * wave per (chain, 16-column tile) walking the steps backwards from strided clean
 * checkpoints; at most 512 packed documents and four views); anything else is
 * BDGDN_ERR_UNSUPPORTED.  The block-form kernels are deterministic, grouped value heads
 * included (dq, dk of a q/k head summed over its v-heads in a fixed order).  The per-step
 * backward sums dq, dk, dg and dbeta over its column tiles with floating-point atomics
 * (summation order not fixed).
 * Range: do, don and the state gradients enter the products as fp16 operands.  Every result
 * is linear in do, don and dht, so the call first finds the largest |entry| of do, don (of
 * every view) and dht on the device, multiplies them by the power of two sigma that puts it
 * in [4, 8) as they are converted, and divides every fp32 result by sigma (exact): upstream
 * gradients of any magnitude (a loss averaged over many tokens, or a large one) keep the
 * fp16 operands' relative precision, and scaling the upstream gradients by a power of two
 * scales every result by exactly that factor.  Non-finite upstream gradients give sigma = 1.
 */
int bdgdn_bwd_train(const bdgdn_fwd_desc_t *desc,
                    const void *q, const void *k, const void *v,
                    const float *g, const float *beta,
                    const void *qn, const void *kn, const void *vn,
                    const float *gn, const float *betan,
                    const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                    const float *h0, const void *do_, const void *don, const float *dht,
                    float *dq, float *dk, float *dv, float *dg, float *dbeta,
                    float *dqn, float *dkn, float *dvn, float *dgn, float *dbetan, float *dh0,
                    void *workspace, size_t workspace_bytes, void *stream);

/* One noisy view of the complementary-view backward: its inputs (as bdgdn_noisy_view_t),
 * the upstream gradient of its readout and its gradients (as dqn .. dbetan of
 * bdgdn_bwd_train). */
typedef struct {
    const void *q, *k, *v;   /* [B*T][h_qk or h_v][d] of desc->dtype, 16-byte aligned      */
    const float *g, *beta;   /* [B*T][h_v] fp32                                              */
    const void *do_;         /* [B*T][h_v][d_v] of desc->out_dtype, 16-byte aligned          */
    float *dq, *dk;          /* [B*T][h_qk][d_k] fp32                                        */
    float *dv;               /* [B*T][h_v][d_v] fp32                                         */
    float *dg, *dbeta;       /* [B*T][h_v] fp32                                              */
} bdgdn_noisy_view_grad_t;

/* Bytes of device workspace bdgdn_bwd_train_views needs (that of bdgdn_bwd_train: the views
 * share it). */
size_t bdgdn_bwd_train_views_workspace(const bdgdn_fwd_desc_t *desc);

/*
 * Backward of bdgdn_fwd_train_views (the complementary-view objective of Sec. 3.3 "Training
 * Objective and Mask Design": several noisy views, each block seeded from the same clean
 * state): the gradients of
 *     sum <do, o> + sum_i sum <views[i].do_, o_i> + <dht, ht>
 * for 1 <= n_views <= 16.  Every view's noisy block b sends its seed's gradient into the
 * clean state gradient at the end of clean block b - 1 (eq. dh-block-recursion, summed over
 * the views).  Clean inputs, h0, do, dht, dq .. dbeta, dh0 and the workspace as for
 * bdgdn_bwd_train; each view's gradients go to its own arrays.  The same support and
 * errors as bdgdn_bwd_train; deterministic except for the grouped-head atomics described
 * there.
 */
int bdgdn_bwd_train_views(const bdgdn_fwd_desc_t *desc,
                          const void *q, const void *k, const void *v,
                          const float *g, const float *beta,
                          const bdgdn_noisy_view_grad_t *views, int32_t n_views,
                          const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                          const float *h0, const void *do_, const float *dht,
                          float *dq, float *dk, float *dv, float *dg, float *dbeta, float *dh0,
                          void *workspace, size_t workspace_bytes, void *stream);

/*
 * One Diffusion-Trust denoise pass over R blocks (Appendix "Per-block denoise loop",
 * "Differences between the denoise pass and the state-update pass").  Request r's
 * block is seeded with state_pool[slot[r]] (slot == NULL means slot[r] = r) and every
 * position reads the block-end state.  state_pool is only read.
 *
 *   state_pool  [n_slots][h_v][d_k][d_v] fp32 (device)
 *   slot        [R] int32 device array of pool indices, or NULL
 *   q, k, v     [R*L][h][d] (dtype); g, beta [R*L][h_v] fp32
 *   o           [R*L][h_v][d_v] block-end readout (out_dtype)
 * Slot indices are not range-checked on the device; they must be valid.
 */
int bdgdn_denoise_step(const bdgdn_serve_desc_t *desc, const float *state_pool,
                       const int32_t *slot, const void *q, const void *k, const void *v,
                       const float *g, const float *beta, void *o, void *stream);

/*
 * Token-causal state-update pass over R blocks (Appendix Algorithm "Diffusion-Trust
 * serving loop", the forward that writes S back): state_pool[slot[r]] is advanced by
 * the L tokens of request r, in place.  o_causal ([R*L][h_v][d_v], out_dtype) receives the
 * causal readout when not NULL.  Slots must be distinct (calls with repeated slots
 * race) and valid.
 */
int bdgdn_commit(const bdgdn_serve_desc_t *desc, float *state_pool, const int32_t *slot,
                 const void *q, const void *k, const void *v,
                 const float *g, const float *beta, void *o_causal, void *stream);

/*
 * The AR-Trust verify pass with its state cache (Appendix "Serving-system machinery for
 * the hybrid backbone", cache-and-scatter; Algorithm "AR-Trust serving round"): the
 * commit pass of bdgdn_commit over each request's block of L = desc->block positions
 * (e.g. the anchor and K draft tokens, L = K + 1), which also writes, for the block's
 * last n_record positions p = L - n_record + i (i = 0 .. n_record-1), the state before
 * position p:
 *
 *   states      [R][n_record][h_v][d_k][d_v] fp32 (device, 16-byte aligned), written
 *               whole; states[r][i] is the state after the first L - n_record + i
 *               positions of request r (the cached state itself when that is 0).
 *
 * The pool then holds the state after all L positions, exactly as after bdgdn_commit
 * (o_causal as there).  1 <= n_record <= block.  Available for bf16 inputs with
 * d_k = d_v = 128 and blocks of at most 32 positions (else BDGDN_ERR_UNSUPPORTED).
 */
int bdgdn_commit_record(const bdgdn_serve_desc_t *desc, float *state_pool, const int32_t *slot,
                        const void *q, const void *k, const void *v,
                        const float *g, const float *beta, void *o_causal,
                        int32_t n_record, float *states, void *stream);

/*
 * The accept step after a verify decision: request r keeps the state at its accepted
 * offset, state_pool[slot[r]][h] = states[r][accept[r]][h] for every v-head h, in one
 * launch (one workgroup per (request, v-head)).
 *
 *   accept      [R] int32 device array; accept[r] == n_record keeps the state already in
 *               the pool (the verify pass's final state); values outside [0, n_record]
 *               also leave the slot untouched (they are not checked on the host).
 *   states      as written by bdgdn_commit_record with the same n_record and desc.
 * state_pool and states must be 16-byte aligned.  Any supported (d_k, d_v).
 */
int bdgdn_accept_states(const bdgdn_serve_desc_t *desc, float *state_pool, const int32_t *slot,
                        const float *states, int32_t n_record, const int32_t *accept, void *stream);

/*
 * The two-stream 1D causal ShortConv in front of the GDR inputs (Appendix "ShortConv under
 * two-stream training", eq. short-conv-clean and eq. short-conv-noisy, computed in the fused
 * form that picks each lag's stream in place), per channel c with filter w[c][0..W-1]:
 *
 *   y[t]   = act(bias[c] + sum_i w[c][i] x[t-i])
 *   yn[t]  = act(bias[c] + sum_i w[c][i] z(t, t-i)),  z(t, s) = xn[s] if s lies in t's
 *            diffusion block, else x[s]
 *
 * with diffusion blocks of `block` rows counted from each sequence's (or document's) start,
 * and rows before that start read as zero (Appendix "Document-packed training", the
 * ShortConv lag mask).  act is the identity or silu.
 *
 *   x, xn, y, yn   [B*T][channels] of dtype (the clean and noisy streams), 8-byte aligned
 *   w              [channels][width] fp32, w[c][i] the weight of lag i
 *   bias           [channels] fp32, or NULL for none
 *   cu_seqlens_*   both NULL (B sequences of T rows) or both [N+1] int32 offsets into the
 *                  packed rows (B == 1, cu[0] == 0, cu[N] == T, non-decreasing; any
 *                  document lengths).  The two copies must hold the same values.
 * Supported: dtype bf16 or fp32, 1 <= width <= 4, channels a multiple of 4 (bf16) or 2
 * (fp32); else BDGDN_ERR_UNSUPPORTED.  The token tensors may be NULL when B*T == 0.
 * Results are deterministic.
 */
typedef enum { BDGDN_ACT_NONE = 0, BDGDN_ACT_SILU = 1 } bdgdn_act_t;

typedef struct {
    int32_t batch;      /* B sequences; must be 1 when packed (num_seqs > 0)           */
    int32_t seqlen;     /* T rows per sequence, or total packed rows                    */
    int32_t num_seqs;   /* N packed documents, 0 when not packed                        */
    int32_t channels;   /* D, the row length of every token tensor                      */
    int32_t width;      /* W filter taps                                                */
    int32_t block;      /* diffusion block size L                                       */
    int32_t activation; /* bdgdn_act_t                                                  */
    int32_t dtype;      /* bdgdn_dtype_t of x, xn, y, yn, dy, dyn, dx, dxn              */
} bdgdn_conv_desc_t;

/* Forward: writes every row of y and yn. */
int bdgdn_shortconv_fwd(const bdgdn_conv_desc_t *desc, const void *x, const void *xn, const float *w,
                        const float *bias, const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                        void *y, void *yn, void *stream);

/* Bytes of device workspace bdgdn_shortconv_bwd needs (0 when there are no rows, or for a
 * descriptor it would reject). */
size_t bdgdn_shortconv_bwd_workspace(const bdgdn_conv_desc_t *desc);

/*
 * Backward of bdgdn_shortconv_fwd for the upstream gradients dy, dyn ([B*T][channels],
 * dtype): writes dx, dxn (dtype, every row), dw ([channels][width] fp32) and, when not
 * NULL, dbias ([channels] fp32); all are overwritten, not accumulated into.  Each noisy
 * output's gradient flows to the stream it read at each lag.  workspace: device memory
 * of at least bdgdn_shortconv_bwd_workspace(desc) bytes, 256-byte aligned, scratch owned
 * by the call until the stream passes it.
 */
int bdgdn_shortconv_bwd(const bdgdn_conv_desc_t *desc, const void *x, const void *xn, const float *w,
                        const float *bias, const void *dy, const void *dyn, const int32_t *cu_seqlens_dev,
                        const int32_t *cu_seqlens_host, void *dx, void *dxn, float *dw, float *dbias,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * bdgdn_shortconv_bwd without a workspace argument, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving or training loops, harnesses that
 * forbid allocation).  It computes exactly what bdgdn_shortconv_bwd computes, with the same
 * kernels and the same summation order (bit-identical results), and calls no allocating
 * routine: its dw / dbias partials live in a scratch array of BDGDN_NOALLOC_SCRATCH_BYTES
 * that the library holds on each GPU it runs on until the process ends (looked up on the
 * first call on a device; the stream's device, or the current device for a NULL stream).
 * Inputs needing more than that (bdgdn_shortconv_bwd_workspace(desc) bytes: 4 (width + 1)
 * channels bytes per started group of 1024 rows, e.g. 1.9 MiB for 16384 rows of 6144
 * channels at width 4) return BDGDN_ERR_SCRATCH before anything is launched.  Every call on one GPU
 * shares that GPU's scratch: calls whose execution overlaps on one GPU (different streams,
 * or threads launching concurrently) race and give undefined dw / dbias; serialise them
 * on one stream.  The caller still owns every input and output buffer.
 */
#define BDGDN_NOALLOC_SCRATCH_BYTES (32u << 20)
int bdgdn_shortconv_bwd_noalloc(const bdgdn_conv_desc_t *desc, const void *x, const void *xn, const float *w,
                                const float *bias, const void *dy, const void *dyn,
                                const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host, void *dx,
                                void *dxn, float *dw, float *dbias, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* BDGDN_H */
