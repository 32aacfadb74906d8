/*
 * lstm_sd.h -- C ABI of a structured-dropout LSTM training step for AMD
 * Instinct MI355X (gfx950).
 *
 * The method (Sec. 3 of "Structured in Space, Randomized in Time: Leveraging
 * Dropout in RNNs for Efficient Training"): dropout masks are drawn per
 * neuron and per time step and shared by every row of the batch (Case-III,
 * Sec. 3.1).  A dropped input or recurrent neuron is then a whole row of the
 * contraction dimension of the gate products (Eq. 1-4), so the forward
 * products run on compacted operands (Sec. 3.2, FP paragraph), the input
 * gradients of Eq. 10 are computed only for kept columns (BP paragraph) and
 * the weight gradients of Eq. 11 only for kept rows (WG paragraph).
 *
 * Conventions shared by every entry point
 *   - L layers, D directions (1 or 2), input dim I, hidden H, batch B,
 *     sequence length T.  K_in(l) = I for l = 0, D*H above.
 *   - Row-vector convention of Eq. 1-4: gate pre-activations a = x W + h U + b
 *     with the 4H gate columns ordered i | f | g | o.
 *   - W[l*D+d] is [K_in(l)][4H] and U[l*D+d] is [H][4H], row-major
 *     ("K-major": a dropped input neuron k is the whole row k).
 *     b[l*D+d] is [4H] float.
 *   - Sequences are time-major: x is [T][B][I], y is [T][B][D*H].
 *   - dtype 0: every tensor is float32.  dtype 1: x, W, U and h0 are
 *     bfloat16 (raw 16-bit words); products accumulate in float32; c0, b, y,
 *     hT, cT, dy and every gradient stay float32.
 *   - Inverted dropout: a kept value is scaled by s = 1/(1-p) (s = 1 when
 *     p = 0).  The non-recurrent (NR) mask of layer l multiplies that
 *     layer's input (shared by both directions); the recurrent (RH) mask of
 *     (l, d) multiplies only the copy of h_prev that enters U.  The cell
 *     state is never dropped.
 *   - compact = 1 skips dropped rows/columns (the method); compact = 0 runs
 *     the same kernels over every row with the mask applied as a
 *     multiplier (the dense baseline).  Both give the same result up to
 *     floating-point summation order.  The weight gradients (bf16) sum every
 *     step with each row multiplied by its mask byte in both modes: on this
 *     device that is faster than the row-sparse form of Eq. 11, which the
 *     environment selects with LSTM_SD_WGRAD_ROWSPARSE=1 (batch <= 32) or
 *     LSTM_SD_WGRAD_GEMM=0 (batch > 32); the result is the same.
 *   - Optional per-row lengths [B] (int32, device): rows freeze h and c and
 *     output 0 from t = lengths[b] on; lengths outside [0, T] are clamped.
 *
 * Ownership and synchronisation
 *   The caller owns every buffer.  All pointers named "device" are device
 *   memory of the current HIP device, 16-byte aligned.  The library
 *   allocates nothing.  Every call only enqueues work on `stream` (a
 *   hipStream_t; NULL = the default stream) and returns; nothing inside a
 *   call waits for the device, so calls can be captured into a HIP graph.
 *   Calls that share a mask, reserve or workspace buffer must be ordered on
 *   one stream.
 *
 * Errors
 *   Every int-returning entry point returns LSTM_SD_OK (0) or a negative
 *   code and then leaves a message for lstm_sd_last_error().  Arguments are
 *   validated before any device work is enqueued.
 */
#ifndef LSTM_SD_H
#define LSTM_SD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LSTM_SD_OK            0
#define LSTM_SD_EINVAL       -1   /* null required pointer, bad dimension, p outside [0,1) */
#define LSTM_SD_EUNSUPPORTED -2   /* dtype or a size beyond the library's limits */
#define LSTM_SD_EHIP         -3   /* HIP launch/runtime error; message has the HIP error string */
#define LSTM_SD_EWORKSPACE   -4   /* a buffer is smaller than its size query returned */

#define LSTM_SD_DTYPE_F32  0
#define LSTM_SD_DTYPE_BF16 1

/* Limits: every K dimension (I, D*H, H) is at most LSTM_SD_MAX_K. */
#define LSTM_SD_MAX_K 2048

typedef struct {
    int32_t num_layers;   /* L >= 1 */
    int32_t input_dim;    /* I >= 1 */
    int32_t hidden;       /* H >= 1 */
    int32_t batch;        /* B >= 1 */
    int32_t seq_len;      /* T >= 1 */
    int32_t num_dirs;     /* D in {1, 2} */
    int32_t dtype;        /* LSTM_SD_DTYPE_F32 or LSTM_SD_DTYPE_BF16 */
    int32_t compact;      /* 1 = skip dropped rows (method), 0 = dense baseline */
    double p_nr;          /* non-recurrent dropout rate, [0, 1) */
    double p_rh;          /* recurrent dropout rate, [0, 1) */
    /* Per-layer rates (a dropout vector with one rate per site, as AWD-LSTM
     * uses, Sec. 4.1): NULL, or a host array of L rates in [0, 1) that
     * replaces p_nr (the NR rate of layer l's input) or p_rh (the RH rate of
     * both directions of layer l).  Read during each call only. */
    const double* p_nr_layer;
    const double* p_rh_layer;
} lstm_sd_dims;

/* Host arrays of L*D device pointers, index l*D + d. */
typedef struct {
    const void* const* W;    /* [K_in(l)][4H], dtype */
    const void* const* U;    /* [H][4H], dtype */
    const float* const* b;   /* [4H] */
} lstm_sd_weights;

/* Host arrays of L*D device pointers, index l*D + d; float32, overwritten. */
typedef struct {
    float* const* dW;        /* [K_in(l)][4H] */
    float* const* dU;        /* [H][4H] */
    float* const* db;        /* [4H] */
} lstm_sd_grads;

/* Byte offsets of the parts of a mask buffer (all relative to its start).
 * Sites: the NR site of layer l is site l; the RH site of (l, d) is site
 * L + l*D + d.  Site s has K(s) neurons (K_in(l) for NR, H for RH); rows are
 * padded to kmax entries.
 *   mask  uint8 [sites][T][kmax]  1 = kept, 0 = dropped
 *   keep  int32 [sites][T][kmax]  ascending kept indices (compact = 1) or
 *                                 0..K(s)-1 (compact = 0); entries past the
 *                                 count are unspecified
 *   pos   int32 [sites][T][kmax]  inverse of keep: position of neuron k in
 *                                 keep, or -1 if k is not listed
 *   count int32 [sites][T]        number of listed entries
 *   drop  int32 [sites][T][kmax]  ascending dropped indices (compact = 1);
 *                                 empty when compact = 0
 *   dcount int32 [sites][T]       number of entries of drop
 *   kseg  int32 [sites][T][17]    kseg[x] = number of kept neurons below
 *                                 floor(x*K(s)/16), x = 0..16: the keep list
 *                                 split into 16 segments of neuron indices
 *   dseg  int32 [sites][T][17]    the same for the drop list */
typedef struct {
    int32_t sites;
    int32_t kmax;
    int32_t seq_len;
    int32_t reserved;
    size_t mask_off, keep_off, pos_off, count_off, drop_off, dcount_off, kseg_off, dseg_off,
        total_bytes;
} lstm_sd_mask_layout;

int         lstm_sd_version(void);
const char* lstm_sd_last_error(void);

/* Size queries; return 0 (and set the error) for invalid dims. */
size_t lstm_sd_mask_bytes(const lstm_sd_dims* dims);
size_t lstm_sd_reserve_bytes(const lstm_sd_dims* dims);
size_t lstm_sd_workspace_bytes(const lstm_sd_dims* dims);
int    lstm_sd_mask_layout_get(const lstm_sd_dims* dims, lstm_sd_mask_layout* out);

/* Draw the Case-III masks of every site for one training step (Sec. 3.1:
 * structured within the batch, fresh at every time step) and build the keep
 * lists ("matrix compaction", Sec. 4).  Neuron k of a site with stream id
 * `sid` at time t is dropped iff the 64-bit word number k%4 of
 * Philox4x64-10(key = (seed, 0), counter = (k/4, t, sid, step)) is below
 * floor(p * 2^64).  Stream ids: NR of layer l = 4l; RH of (l, d) = 4l+2+d.
 * mask_buf: device, lstm_sd_mask_bytes(dims) bytes. */
int lstm_sd_mask_generate(const lstm_sd_dims* dims, uint64_t seed, uint64_t step,
                          void* mask_buf, size_t mask_bytes, void* stream);

/* Case-IV masks (Sec. 3, the most restrictive case: structured in the batch
 * and the same at every time step; the paper keeps Case-III because this one
 * varies too little): one draw per site for the whole sequence, the draw of
 * t = 0 of lstm_sd_mask_generate, repeated at every t, with its keep lists.
 * Every other entry point takes the result unchanged.  For comparing the
 * cost of per-t randomness. */
int lstm_sd_mask_generate_fixed(const lstm_sd_dims* dims, uint64_t seed, uint64_t step,
                                void* mask_buf, size_t mask_bytes, void* stream);

/* The compaction step alone ("matrix compaction", Sec. 4) on masks the
 * caller wrote: rebuild keep, pos, count, drop, dcount, kseg and dseg from
 * the mask bytes already in mask_buf (one Case-III row per site and t,
 * Sec. 3.1), e.g. to force a pattern such as a step with every neuron
 * dropped.  mask_buf: device, lstm_sd_mask_bytes(dims) bytes. */
int lstm_sd_mask_compact(const lstm_sd_dims* dims, void* mask_buf, size_t mask_bytes,
                         void* stream);

/* Forward unroll, Eq. 1-6 with the masks of mask_buf.
 *   x        device [T][B][I], dtype
 *   lengths  device [B] int32, or NULL (every row has length T)
 *   h0       device [L*D][B][H], dtype;  c0 device [L*D][B][H] float
 *   y        device [T][B][D*H] float: top layer output (0 at padded steps)
 *   hT, cT   device [L*D][B][H] float: state after the last valid step
 *   reserve  device, lstm_sd_reserve_bytes(dims): activations kept for
 *            lstm_sd_backward
 *   workspace device, lstm_sd_workspace_bytes(dims) */
int lstm_sd_forward(const lstm_sd_dims* dims, const lstm_sd_weights* w,
                    const void* x, const int32_t* lengths,
                    const void* h0, const float* c0,
                    const void* mask_buf, size_t mask_bytes,
                    float* y, float* hT, float* cT,
                    void* reserve, size_t reserve_bytes,
                    void* workspace, size_t workspace_bytes, void* stream);

/* Back-propagation through time, Eq. 7-11, for the forward pass that filled
 * `reserve` (same dims, weights, x, lengths, h0, c0 and masks).
 *   dy       device [T][B][D*H] float: dLoss/dy
 *   dhT, dcT device [L*D][B][H] float, or NULL for zero
 *   dx       device [T][B][I] float, or NULL to skip the input gradient of
 *            layer 0; dropped columns are written as exact zeros
 *   dh0, dc0 device [L*D][B][H] float
 *   g        gradients, overwritten (rows of never-kept neurons are 0) */
int lstm_sd_backward(const lstm_sd_dims* dims, const lstm_sd_weights* w,
                     const void* x, const int32_t* lengths,
                     const void* h0, const float* c0,
                     const void* mask_buf, size_t mask_bytes,
                     const void* reserve, size_t reserve_bytes,
                     const float* dy, const float* dhT, const float* dcT,
                     float* dx, float* dh0, float* dc0, const lstm_sd_grads* g,
                     void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * forward pass of lstm_sd_forward with the same arguments except the
 * workspace, which the library holds itself in a file-scope device array of
 * LSTM_SD_STATIC_WORKSPACE_MAX bytes (each GPU the library runs on holds one
 * until the process ends).  The call allocates nothing; the caller still
 * owns the mask, reserve and output buffers, and `reserve` feeds
 * lstm_sd_backward (with a workspace of the caller's) as after
 * lstm_sd_forward.  Dims whose lstm_sd_workspace_bytes exceeds the maximum
 * are rejected with LSTM_SD_EUNSUPPORTED before any device work.  Every call
 * on one GPU uses the same array, and the pass clears what it needs cleared
 * in its first kernel: calls that overlap on one GPU (other streams, other
 * threads) race, so order them on one stream.  A barrier time-out is visible
 * as NaN in hT, cT and y (there is no workspace to pass to lstm_sd_status). */
#define LSTM_SD_STATIC_WORKSPACE_MAX ((size_t)64 << 20)
int lstm_sd_forward_static(const lstm_sd_dims* dims, const lstm_sd_weights* w,
                           const void* x, const int32_t* lengths,
                           const void* h0, const float* c0,
                           const void* mask_buf, size_t mask_bytes,
                           float* y, float* hT, float* cT,
                           void* reserve, size_t reserve_bytes, void* stream);

/* Mean-squared-error loss of y against target over valid (t, b) and all
 * D*H features, and its gradient: loss = sum (y-target)^2 / N,
 * dy = 2 (y - target) / N at valid positions and 0 elsewhere, with N =
 * (number of valid (t, b)) * D*H.  A loss of the workloads, not of the
 * paper (its tasks need datasets).
 *   y, target  device [T][B][D*H] float;  lengths device [B] or NULL
 *   dy         device [T][B][D*H] float (written)
 *   loss       device float[1] (written)
 *   workspace  device, lstm_sd_workspace_bytes(dims); only its last 16 KiB
 *              are used, so the same buffer can be shared with the step. */
int lstm_sd_mse_grad(const lstm_sd_dims* dims, const float* y, const float* target,
                     const int32_t* lengths, float* dy, float* loss,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Embedding-table gradient of a language model whose layer-0 input is an
 * embedding lookup, x_t[b] = E[tokens[t][b]]: the step just below the path.
 * Row v of d_emb receives the sum of the layer-0 input gradient rows dx_t[b]
 * over every (t, b) with tokens[t][b] = v, over the columns kept at t (layer
 * 0's NR mask; dx is zero in the dropped columns, Eq. 10, and they are not
 * accumulated).  Each row's sum is formed in a fixed order (four partial
 * sums over interleaved groups of 64 positions, each ascending, then added in
 * group order) and added to d_emb once: deterministic, no atomics on d_emb.
 *   tokens   device [T][B] int32; ids outside [0, vocab) are skipped
 *   vocab    rows of the table (> 0)
 *   dx       device [T][B][I] float: lstm_sd_backward's dx
 *   mask_buf device, the masks of the step (as for lstm_sd_backward)
 *   d_emb    device [vocab][I] float, accumulated into (+=): rows of tokens
 *            that occur change, the others are not touched
 * Errors: LSTM_SD_EINVAL (null pointer, vocab <= 0, bad dims),
 * LSTM_SD_EWORKSPACE (mask_bytes too small), LSTM_SD_EHIP. */
int lstm_sd_embedding_backward(const lstm_sd_dims* dims, const int32_t* tokens, int vocab, const float* dx,
                               const void* mask_buf, size_t mask_bytes, float* d_emb, void* stream);

/* ---------------------------------------------------------------------------
 * Output head of a language model: structured dropout on the top LSTM
 * output before the FC (vocabulary projection) layer, the FC layer, and the
 * softmax cross-entropy loss.  The paper's timings include the FC layers'
 * products after compaction (Sec. 4, experimental setup); its language
 * models drop the LSTM output before the FC layer (Sec. 4.1) and its
 * translation models the final encoder/decoder outputs, the projection being
 * sized by the vocabulary (Sec. 4.2).  A Case-III mask on the FC input
 * (Sec. 3.1) propagates as in Sec. 3.2 for one product: the forward product
 * reads only the kept input columns, the input gradient is written only in
 * the kept columns, and the weight gradient only in the rows kept at each t.
 *   z[t][b] = (s * m[t] * y[t][b]) W + c,   s = 1/(1-p_out)
 *   loss    = mean over rows that count of logsumexp(z) - z[target]
 * A row (t, b) counts when t < lengths[b] and its target is in [0, vocab)
 * (other targets act as an ignore index). */
typedef struct {
    int32_t features;     /* F = D*H of the LSTM below, 1 .. LSTM_SD_MAX_K */
    int32_t vocab;        /* V >= 4, a multiple of 4; F*V*sizeof(dtype) < 2^31 */
    int32_t batch;        /* B, as the LSTM */
    int32_t seq_len;      /* T, as the LSTM */
    int32_t dtype;        /* LSTM_SD_DTYPE_F32 or LSTM_SD_DTYPE_BF16 */
    int32_t compact;      /* 1 = skip dropped rows (method), 0 = dense baseline */
    int32_t stream_id;    /* mask stream of the output site: 4*L for an L-layer stack */
    int32_t reserved;
    double p_out;         /* output dropout rate, [0, 1) */
} lstm_sd_head_dims;

/* Sizes (0 and the error set for invalid dims).  The head's mask buffer has
 * the layout of lstm_sd_mask_layout with one site of K = features. */
size_t lstm_sd_head_mask_bytes(const lstm_sd_head_dims* hd);
size_t lstm_sd_head_workspace_bytes(const lstm_sd_head_dims* hd);
int    lstm_sd_head_mask_layout_get(const lstm_sd_head_dims* hd, lstm_sd_mask_layout* out);

/* Draw the output site's mask for one training step with the generator of
 * lstm_sd_mask_generate (stream id hd->stream_id, rate p_out). */
int lstm_sd_head_mask_generate(const lstm_sd_head_dims* hd, uint64_t seed, uint64_t step,
                               void* mask_buf, size_t mask_bytes, void* stream);

/* Forward: logits of every (t, b).
 *   W_fc     device [F][V], dtype (input-major, as the LSTM weights)
 *   b_fc     device [V] float
 *   y        device [T][B][F] float: the top LSTM output (lstm_sd_forward's y)
 *   logits   device [T][B][V] float (written)
 *   workspace device, lstm_sd_head_workspace_bytes(hd); it carries the
 *            forward's prepared input to lstm_sd_head_backward, so the same
 *            buffer must reach the backward unchanged. */
int lstm_sd_head_forward(const lstm_sd_head_dims* hd, const void* W_fc, const float* b_fc, const float* y,
                         const void* mask_buf, size_t mask_bytes, float* logits, void* workspace,
                         size_t workspace_bytes, void* stream);

/* Loss and backward of the head.
 *   targets  device [T][B] int32;  lengths device [B] int32 or NULL
 *   logits   device [T][B][V] float from lstm_sd_head_forward
 *   loss     device float[1] (written): the mean cross-entropy (0 if no row counts)
 *   dy       device [T][B][F] float (written): the gradient for the top LSTM
 *            output, zero in the columns dropped at t (feed it to
 *            lstm_sd_backward as dy)
 *   dW_fc    device [F][V] float (overwritten): zero in rows never kept
 *   db_fc    device [V] float (overwritten)
 * Errors: LSTM_SD_EINVAL, LSTM_SD_EUNSUPPORTED, LSTM_SD_EWORKSPACE, LSTM_SD_EHIP. */
int lstm_sd_head_backward(const lstm_sd_head_dims* hd, const void* W_fc, const int32_t* targets,
                          const int32_t* lengths, const void* mask_buf, size_t mask_bytes, const float* logits,
                          float* loss, float* dy, float* dW_fc, float* db_fc, void* workspace,
                          size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Case-I dropout, the comparator of the paper's "NR+Random" baselines (Sec. 3,
 * Sec. 4): an unstructured mask, one keep bit per element (t, b, k) of a layer
 * input, so no row of a product can be skipped; the step then runs dense.
 * Element (t, b, k) is dropped iff word k%4 of Philox4x64-10(key = (seed, 0),
 * counter = (k/4, t, stream_id + 2^32 (b+1), step)) is below floor(p * 2^64)
 * (the Case-III generator with the batch row in the stream's high word).
 *   src   device [T][B][K], src_dtype;  dst device [T][B][K], dst_dtype:
 *         dst = src * kept / (1-p)
 *   mask  device [T][B][K] uint8 (written): 1 = kept
 * A stack of L layers takes one call per layer input (stream 4l for layer l,
 * as the Case-III NR site) and a single-layer dense step per layer. */
int lstm_sd_case1_dropout(int32_t seq_len, int32_t batch, int32_t features, int32_t src_dtype, const void* src,
                          int32_t dst_dtype, void* dst, uint8_t* mask, uint64_t seed, uint64_t step,
                          int32_t stream_id, double p, void* stream);

/* The gradient through lstm_sd_case1_dropout: dsrc = dx * mask / (1-p).
 *   dx, dsrc  device [T][B][K] float (may alias);  mask as written by the forward */
int lstm_sd_case1_dropout_backward(int32_t seq_len, int32_t batch, int32_t features, const float* dx,
                                   const uint8_t* mask, double p, float* dsrc, void* stream);

/* Failure of a step's persistent kernels.  The recurrences run as persistent
 * launches whose workgroups meet at a grid barrier once per time step (one
 * step of Eq. 1-6 forward, of Eq. 7-10 backward, needs the whole h_{t-1} or
 * DA of the step before).  Every barrier wait is bounded by wall-clock time
 * (0.5 s by default); a wait that times out stops its launch, and then:
 *   - the forward writes NaN into hT, cT and every step of y;
 *   - the backward writes NaN into dh0, dc0, dx and every weight and bias
 *     gradient (also when it was the forward of the same step that failed);
 *   - the pass bit (1 = forward, 2 = backward) is ORed into a status word in
 *     the workspace, which lstm_sd_forward's first kernel clears.
 * lstm_sd_status waits for `stream` (a host synchronisation: not for graph
 * capture) and returns LSTM_SD_EHIP with a message naming the failed pass
 * when the status word of `workspace` is set since the last lstm_sd_forward
 * on it, else LSTM_SD_OK.  A time-out cannot happen while the grid runs
 * alone on the device; it guards against a device shared with other work.
 * lstm_sd_set_barrier_timeout sets the bound for the whole process: seconds
 * < 0 restores the default; 0 makes every wait fail at once (every kernel
 * still ends normally), to exercise this path from the host. */
int lstm_sd_status(const lstm_sd_dims* dims, const void* workspace, size_t workspace_bytes, void* stream);
int lstm_sd_set_barrier_timeout(double seconds);

/* Instrumentation for measuring one kernel's average duration on the
 * stream it runs on.  After lstm_sd_kernel_timer_start(name), every launch
 * of the named kernel made by this library is bracketed by a pair of HIP
 * events recorded on its launch stream; lstm_sd_kernel_timer_stop()
 * waits for the last pair, returns the summed elapsed time in milliseconds
 * and the number of launches, and turns the timer off.  Names:
 * "mask_build", "transpose", "fx", "step", "bwd", "dx", "wgrad",
 * "fwd_persist", "bwd_persist" (the persistent recurrent kernels: one launch
 * per layer, or one for a whole unidirectional stack),
 * "emb_grad" (lstm_sd_embedding_backward's one kernel), "ce" (the head's
 * softmax cross-entropy kernels; the head's FC products count as "fx", "dx"
 * and "wgrad").  Events
 * are created by the library (no device memory is allocated).  Not
 * thread-safe; for benchmarks. */
int lstm_sd_kernel_timer_start(const char* kernel);
int lstm_sd_kernel_timer_stop(double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* LSTM_SD_H */
