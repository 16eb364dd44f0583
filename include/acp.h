/*
 * acp.h - C ABI of the ACP-SGD gradient compressor for AMD Instinct MI355X (gfx950).
 *
 * ACP-SGD ("alternate compressed Power-SGD", arXiv 2306.08881, Section IV-A,
 * Algorithms 1 and 2) compresses every gradient matrix M_t (n x m) of a model
 * to one rank-r factor per step, alternating by the parity of the step t:
 *
 *   odd t  (P-step): Q_t = orth(Q_{t-1});  P_t = (M_t + E_{t-1}) Q_t;
 *   even t (Q-step): P_t = orth(P_{t-1});  Q_t = (M_t + E_{t-1})^T P_t;
 *   both:            E_t = M_t + E_{t-1} - P_t Q_t^T   (local factor, before the all-reduce)
 *                    the new factor (P_t or Q_t) is all-reduced (summed over p workers)
 *                    and the step returns M_hat_t = P_t Q_t^T / p with the aggregated factor.
 *
 * orth() is the Gram-Schmidt factor: thin QR with a positive diagonal R; a
 * column whose residual norm is at most 1e-4 of its norm (or zero) is set to
 * zero.  E_0 = 0 and P_0, Q_0 are i.i.d. standard normal (Section IV-A,
 * "Error-feedback"), drawn by a counter-based generator (see acp_init).
 *
 * Gradients are fused into buckets (Section IV-B, "Tensor Fusion", "Buffer
 * Size"): tensors in reverse registration order, a bucket closes once its
 * byte size reaches the cap (25 MiB by default).  Vector-shaped gradients,
 * and matrices with r >= min(n, m), are not compressed (Section IV-C): they
 * travel raw in the factor buffer.  A tensor of shape (d0, d1, ...) is the
 * matrix n = d0, m = d1 * d2 * ... .
 *
 * Buffers (all fp32, row-major, packed, no padding):
 *   gradient bucket b : grad_elems(b) floats; tensor k of the bucket at grad_off[k].
 *   factor buffer b   : on odd steps factor_elems_p(b) floats (P_t, n x r, per compressed
 *                       tensor at fac_off_p[k]; raw vector at fac_off_p[k]); on even steps
 *                       factor_elems_q(b) floats (Q_t, m x r, at fac_off_q[k]).
 *   output bucket b   : like the gradient bucket; receives M_hat_t (and raw vectors / p).
 *
 * Ownership: the caller owns every device buffer and stream.  The library
 * needs one device block for its state (the error E, the factors, small
 * workspaces and its launch tables); the caller allocates it (acp_state_bytes)
 * and hands it over with acp_bind_state.  The library itself never allocates
 * device memory.  Device pointers must be 16-byte aligned.
 *
 * Sequencing: per bucket, steps run 1, 2, 3, ... and compress(t) must precede
 * decompress(t); anything else returns ACP_E_STEP and changes nothing.
 * Buckets are independent and may be processed on different streams; calls
 * on one bucket must be ordered on the caller's side.  A context is not
 * thread-safe.  All argument, state and sequencing checks run on the host
 * before anything is enqueued.  Kernel launch failures return ACP_E_DEVICE;
 * asynchronous device faults surface at a later HIP call.
 */
#ifndef ACP_H
#define ACP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct acp_ctx acp_ctx;

typedef enum {
  ACP_OK = 0,
  ACP_E_INVALID = -1,     /* bad argument (null, out of range, misaligned, bad shape) */
  ACP_E_STEP = -2,        /* call out of step order */
  ACP_E_STATE = -3,       /* state not bound / wrong size / corrupt checkpoint */
  ACP_E_DEVICE = -4,      /* a HIP call failed */
  ACP_E_UNSUPPORTED = -5  /* valid request the library does not implement */
} acp_status;

/* flags of acp_init */
#define ACP_FLAG_EF 1u            /* error feedback (Algorithm 2); off = Algorithm 1's ACP branch */
#define ACP_FLAG_REUSE 2u         /* reuse the previous factor; off = draw it anew every step */
#define ACP_FLAG_POWERSGD 4u      /* Power-SGD (Algorithm 1, left) through acp_powersgd_* */
#define ACP_FLAGS_DEFAULT 3u

/* which factor for acp_factor / acp_init_factor */
#define ACP_FACTOR_P 0
#define ACP_FACTOR_Q 1

/*
 * acp_init - plan the layout and draw P_0, Q_0 on the host.  No device work (Section IV-B and
 * IV-C for the layout; Section IV-A, "Error-feedback", for E_0 = 0 and P_0, Q_0).  Layout rules:
 * whole tensors in reverse registration order, a bucket closing once its bytes reach the cap;
 * vectors and matrices with r >= min(n, m) pass through raw.  Errors: ACP_E_INVALID for a bad
 * argument (shape, rank, cap, world size, unknown flag), ACP_E_UNSUPPORTED for Power-SGD without
 * reuse.
 *   num_tensors      number of parameters, in registration (forward) order.
 *   ndims[i]         rank of parameter i (1..8); dims holds all dims flattened, each in
 *                    1..2^31.  A compressed matrix (ndims >= 2 and r < min(n, m), n = dim 0,
 *                    m = product of the others) may have at most min(2^24, (2^32 - 1) / (4 r))
 *                    columns m; a longer one returns ACP_E_INVALID.
 *   rank             r: 1, 2, 4, 8, 16, 32, 64, 128 or 256.
 *   seed             key of the initial-factor draw: element i (row-major) of P_0 (f = 0) or
 *                    Q_0 (f = 1) of tensor k is z = sqrt(-2 ln u1) cos(2 pi u2) rounded to fp32,
 *                    with s = mix(seed ^ mix(2k + f)), u1 = ((mix(s + (2i+1)g) >> 11) + 1) 2^-53,
 *                    u2 = (mix(s + (2i+2)g) >> 11) 2^-53, mix the SplitMix64 finaliser and
 *                    g = 0x9E3779B97F4A7C15.
 *   bucket_cap_bytes fusion cap (> 0); 26214400 is PyTorch-DDP's 25 MiB default.
 *   world_size       p >= 1; decompress divides the aggregated sum by p.
 *   flags            ACP_FLAG_*.  Without ACP_FLAG_REUSE (the ablation of Section V-B) every
 *                    step orthogonalises a fresh draw instead of the previous factor: at step t
 *                    the factor is the draw above with the key mix(seed ^ mix(t 2^32 + 2k + f))
 *                    (t = 0 gives P_0, Q_0), made on the device.  ACP_FLAG_POWERSGD selects
 *                    Power-SGD (needs ACP_FLAG_REUSE): such a context takes acp_powersgd_* and
 *                    refuses acp_compress / acp_decompress (ACP_E_UNSUPPORTED), and vice versa.
 * On success *out owns host memory only; free it with acp_destroy.
 */
acp_status acp_init(acp_ctx **out, int32_t num_tensors, const int32_t *ndims, const int64_t *dims,
                    int32_t rank, uint64_t seed, int64_t bucket_cap_bytes, int32_t world_size,
                    uint32_t flags);

/*
 * acp_state_bytes - size in bytes of the device state block the caller must allocate (256-byte
 * aligned): the error E of Algorithm 2 (one fp32 slot per bucket element, Section IV-A
 * "Error-feedback"), the factors P and Q kept from step to step (Section IV-A, query reuse),
 * the orthogonalisation transforms, the Q-step and Gram partial sums and the launch tables.
 * ACP_E_INVALID for a NULL argument.
 */
acp_status acp_state_bytes(const acp_ctx *ctx, int64_t *bytes);

/*
 * acp_bind_state - adopt the caller's device block (>= acp_state_bytes, 256-byte aligned) on
 * the current HIP device.  Uploads P_0, Q_0 and the launch tables, zeroes E and prepares the
 * orthogonalisation of Q_0 for step 1, all on `stream` (a hipStream_t, or NULL for the default
 * stream), then waits for the stream.  Re-binding resets the state to step 0.
 */
acp_status acp_bind_state(acp_ctx *ctx, void *device_ptr, int64_t bytes, void *stream);

/* Number of gradient buckets (Section IV-B, "Buffer Size"), or -1 for a NULL context. */
int32_t acp_num_buckets(const acp_ctx *ctx);

/*
 * acp_bucket_info - bucket b's sizes in elements (any output pointer may be NULL): its tensors,
 * the gradient / output bucket, and the factor buffer of a P-step (each compressed tensor's P,
 * n x r, and every raw vector) and of a Q-step (Q, m x r, and the vectors): what one all-reduce
 * of that bucket carries (Section IV-B, compressed tensors copied into one buffer per bucket).
 * ACP_E_INVALID for a NULL context or b out of range.
 */
acp_status acp_bucket_info(const acp_ctx *ctx, int32_t b, int32_t *num_tensors, int64_t *grad_elems,
                           int64_t *factor_elems_p, int64_t *factor_elems_q);

/*
 * acp_layout - bucket b's metadata, one entry per tensor in bucket order (arrays of
 * num_tensors from acp_bucket_info, owned by the caller; any pointer may be NULL to skip it):
 * registration index, element offsets in the gradient bucket and in the P-step / Q-step factor
 * buffers (packed, no padding), and whether the tensor is compressed.  The layout is the one of
 * Section IV-B ("Buffer Size": whole tensors in backward order, closing at the cap) and IV-C
 * (vectors raw, other tensors reshaped to dim 0 x the rest).  ACP_E_INVALID for a NULL context
 * or b out of range.
 */
acp_status acp_layout(const acp_ctx *ctx, int32_t b, int32_t *tensor_ids, int64_t *grad_off,
                      int64_t *fac_off_p, int64_t *fac_off_q, int32_t *compressed);

/* Per-tensor view: compressed flag, matrix shape n x m (numel x 1 if not compressed), bucket. */
acp_status acp_tensor_info(const acp_ctx *ctx, int32_t tensor_id, int32_t *compressed, int64_t *n,
                           int64_t *m, int32_t *bucket);

/*
 * acp_fusion_groups - compressed-buffer fusion (Section IV-B, "Buffer Size"): what a step sends
 * (which = ACP_FACTOR_P: each compressed tensor's P factor, n x r, as on P-steps;
 * ACP_FACTOR_Q: its Q factor, m x r, as on Q-steps; the raw gradient of every other tensor on
 * both) grouped like the gradient buckets, whole tensors in backward (reverse registration)
 * order, with the bucket cap scaled by that step's compression rate (elements sent over gradient
 * elements).  A group closes once its bytes reach the scaled cap.  group_of (num_tensors entries
 * in registration order, or NULL) receives each tensor's group, 0 being the first group in
 * backward order; *num_groups the number of groups.  Host metadata only: it tells a caller that
 * all-reduces fused factor buffers which tensors travel together; acp_compress and
 * acp_decompress keep one factor buffer per gradient bucket.  ACP_E_INVALID for a NULL ctx or
 * num_groups or another `which`.
 */
acp_status acp_fusion_groups(const acp_ctx *ctx, int32_t which, int32_t *group_of, int32_t *num_groups);

/* Host copy of the initial factor P_0 (which = ACP_FACTOR_P, n*r floats) or Q_0 (m*r floats). */
acp_status acp_init_factor(const acp_ctx *ctx, int32_t tensor_id, int32_t which, float *host_out,
                           int64_t count);

/*
 * acp_compress - step `step` of bucket b (Algorithm 2 up to the all-reduce).  Reads the gradient
 * bucket `grad` (device), updates E in the state and writes the local factors and raw vectors
 * into `factor_buf` (device, factor_elems_p/q(b) floats by parity), enqueued on `stream`.
 * `factor_buf` must not overlap `grad`.  The caller all-reduces (sums) factor_buf across workers.
 * At rank 4 a P-step whose column-class launches are all small may run some of them on a stream
 * the context owns (made at bind on the bound device, default priority), forked from `stream`
 * by an event and joined back into it before the call returns: work enqueued on `stream` after
 * the call, and a graph captured on it, see the whole step.
 */
acp_status acp_compress(acp_ctx *ctx, int64_t step, int32_t b, const float *grad, float *factor_buf,
                        void *stream);

/*
 * acp_compress_noalloc - acp_compress for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  Same checks, same
 * kernels, bitwise the same results and state changes as acp_compress, except that the bucket's
 * Q-step partial sums (the per-row-chunk products that a second kernel adds) go to a static
 * device array of the library instead of the state block: 32 MiB, one copy per GPU, held until
 * the process ends, its address looked up once per device in acp_bind_state.  Nothing is
 * allocated by this call.  A bucket whose partials need more than 32 MiB returns
 * ACP_E_UNSUPPORTED (acp_compress takes it); ACP_E_DEVICE if the array's address could not be
 * looked up.  Every call on one GPU shares that GPU's array and the partials of one call are
 * dead once it is done, so nothing is cleared between calls; calls that overlap on one GPU (on
 * other streams, contexts or threads) race on the array and must be ordered by the caller.
 */
acp_status acp_compress_noalloc(acp_ctx *ctx, int64_t step, int32_t b, const float *grad,
                                float *factor_buf, void *stream);

/*
 * acp_decompress - finish step `step` of bucket b (Algorithm 2, the returned P_t Q_t^T after the
 * all-reduce): from the aggregated (summed) factor buffer `agg_factor` (device), write
 * M_hat = P_t Q_t^T / p for every compressed tensor and raw/p for every vector into `out`
 * (device, grad_elems(b) floats; may alias the gradient bucket but not agg_factor), and keep the
 * aggregated factor as the next step's reused factor (Section IV-A, query reuse).
 * At ranks 8 to 64 the orthogonalisation of that factor (Section IV-A: its Gram, Cholesky and
 * W, and the orthogonal factor the next compress multiplies by) runs on the context's second
 * stream beside the decompress kernel, forked from `stream` and joined back into it before the
 * call returns; the bucket's next compress then skips forming the orthogonal factor itself (it
 * forms it after a fresh bind, a state load, or with fresh draws).
 * ACP_E_STEP unless compress(step) of this bucket came last; ACP_E_INVALID for bad buffers.
 */
acp_status acp_decompress(acp_ctx *ctx, int64_t step, int32_t b, const float *agg_factor, float *out,
                          void *stream);

/*
 * acp_compress_all / acp_decompress_all - the same step for every bucket at once (one launch per
 * kernel kind for up to 64 buckets), as after a backward pass without overlap.  Results are
 * bitwise those of calling acp_compress / acp_decompress for every bucket.  `grads`,
 * `factor_bufs`, `agg_factors` and `outs` are host arrays of acp_num_buckets() device
 * pointers, each with the layout of the per-bucket call.  Every bucket must be ready for the
 * step, else ACP_E_STEP and nothing is enqueued.
 */
acp_status acp_compress_all(acp_ctx *ctx, int64_t step, const float *const *grads,
                            float *const *factor_bufs, void *stream);
/*
 * HIP graphs: the compress and decompress calls enqueue kernels only (no memset, no allocation,
 * no host synchronisation; the fork to the context's stream and the join back are event waits,
 * which capture records), with arguments that depend on the step only through its parity once
 * every bucket has run two steps (with reuse; without it the draw is keyed by the step number).
 * So one odd and one even step's calls may be captured (hipStreamBeginCapture on `stream`) and
 * the two graphs replayed in turn for later steps, with the same buffers.  Capture enqueues
 * nothing and advances the context's host-side step record by the captured steps; replays do not
 * advance it, so calls made after replays see the parity of the last captured step: replay an
 * even number of steps before calling the library again.
 */
acp_status acp_decompress_all(acp_ctx *ctx, int64_t step, const float *const *agg_factors,
                              float *const *outs, void *stream);

/*
 * Power-SGD (Algorithm 1, left) on a context made with ACP_FLAG_POWERSGD, with error feedback
 * applied as Algorithm 2 applies it when ACP_FLAG_EF is set.  Step t of bucket b takes three
 * calls, the caller all-reducing (summing) the buffer the first two write:
 *   acp_powersgd_p          M' = M_t + E_{t-1} (kept in the state for the second half);
 *                           P_t = M' Q_{t-1} into p_buf (P-step layout, factor_elems_p(b)
 *                           floats; raw vectors too).
 *   acp_powersgd_q          P_t = orth(p_agg's P), the all-reduced P; Q_t = M'^T P_t into q_buf
 *                           (Q-step layout, factor_elems_q(b) floats; raw vectors too);
 *                           E_t = M' - P_t Q_t^T with this local Q_t.  `grad` is the same
 *                           gradient bucket as in acp_powersgd_p (read again without error
 *                           feedback).
 *   acp_powersgd_decompress M_hat = P_t Q_agg^T / p into `out`, raw vectors as q_agg / p; Q_agg
 *                           is kept as Q_t, which step t + 1 multiplies by as it is.
 * Q_0 is the same draw as ACP-SGD's.  The calls reuse ACP-SGD's product, orthogonalisation and
 * decompress kernels.  Buffers are device memory, 16-byte aligned; p_buf must not overlap grad,
 * q_buf neither grad nor p_agg, out not q_agg.  Out-of-order calls return ACP_E_STEP; on an
 * ACP-SGD context ACP_E_UNSUPPORTED.  After decompress, acp_factor returns P_t (ACP_FACTOR_P) and
 * Q_agg (ACP_FACTOR_Q), and acp_error E_t; between the first and second half acp_error returns
 * ACP_E_STEP.  The _all forms take host arrays of acp_num_buckets() device pointers and run every
 * bucket in one launch per kernel kind.
 */
acp_status acp_powersgd_p(acp_ctx *ctx, int64_t step, int32_t b, const float *grad, float *p_buf,
                          void *stream);
acp_status acp_powersgd_q(acp_ctx *ctx, int64_t step, int32_t b, const float *grad, const float *p_agg,
                          float *q_buf, void *stream);
acp_status acp_powersgd_decompress(acp_ctx *ctx, int64_t step, int32_t b, const float *q_agg, float *out,
                                   void *stream);
acp_status acp_powersgd_p_all(acp_ctx *ctx, int64_t step, const float *const *grads,
                              float *const *p_bufs, void *stream);
acp_status acp_powersgd_q_all(acp_ctx *ctx, int64_t step, const float *const *grads,
                              const float *const *p_aggs, float *const *q_bufs, void *stream);
acp_status acp_powersgd_decompress_all(acp_ctx *ctx, int64_t step, const float *const *q_aggs,
                                       float *const *outs, void *stream);

/*
 * acp_error - write the current error E of bucket b's compressed tensors into `e_out` (device,
 * laid out like the gradient bucket; vector slots are left untouched).  Does not change the state.
 * ACP_E_UNSUPPORTED without error feedback.
 */
acp_status acp_error(const acp_ctx *ctx, int32_t b, float *e_out, void *stream);

/*
 * acp_factor - copy factor P_t (which = ACP_FACTOR_P, n x r) or Q_t (ACP_FACTOR_Q, m x r) of the
 * last completed step of a compressed tensor into `dev_out` (device).  After an odd step P_t is
 * the aggregated factor and Q_t the orthogonalised one; after an even step the reverse.
 * ACP_E_STEP before step 1 completes.
 */
acp_status acp_factor(const acp_ctx *ctx, int32_t tensor_id, int32_t which, float *dev_out,
                      void *stream);

/*
 * Checkpoint: acp_get_state writes the whole state (step counters, E, factors, orthogonalisation
 * transforms) into a host buffer of acp_checkpoint_bytes; acp_set_state restores it into a bound
 * context built with the same shapes, rank, seed, cap, world size and flags.  Both synchronise
 * the device.  Restoring and continuing is bitwise identical to not stopping.
 */
acp_status acp_checkpoint_bytes(const acp_ctx *ctx, int64_t *bytes);
acp_status acp_get_state(const acp_ctx *ctx, void *host_buf, int64_t bytes);
acp_status acp_set_state(acp_ctx *ctx, const void *host_buf, int64_t bytes);

/*
 * Kernel timing, for benchmarks: acp_profile_start makes every later launch of one kernel family
 * on this context record a HIP event pair on its stream (at most max_launches launches; later
 * ones run untimed); acp_profile_stop waits for those events and returns the number of timed
 * launches, their summed duration in seconds and their summed algorithmic bytes (the data the
 * method must move, excluding any re-reads: 12 B per element of M, E read and E written in a
 * compress kernel, 4 B per element of M_hat, 8 B per raw-vector element, 4 B per factor
 * element read or written).  Events are created in acp_profile_start and destroyed in
 * acp_profile_stop; no device memory is allocated.
 */
#define ACP_KERNEL_P_STEP 1       /* P-step compress kernels */
#define ACP_KERNEL_Q_STEP 2       /* Q-step compress main kernel */
#define ACP_KERNEL_Q_FINISH 3     /* Q-step partial-sum finish */
#define ACP_KERNEL_RECONSTRUCT 4  /* decompress kernels */
#define ACP_KERNEL_ORTH 5         /* separate orthogonalisation kernels (general path, r > 8) */
/* Raw-vector launches of their own (ranks 8 and up) belong to no family; at rank 4 the vectors
 * ride in the P-step, Q-step and decompress launches. */
acp_status acp_profile_start(acp_ctx *ctx, int32_t kernel_family, int32_t max_launches);
acp_status acp_profile_stop(acp_ctx *ctx, int64_t *launches, double *seconds, double *alg_bytes);

/* Text of the last error on this context ("" if none).  Valid until the next call on ctx. */
const char *acp_last_error(const acp_ctx *ctx);

void acp_destroy(acp_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* ACP_H */
