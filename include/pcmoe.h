/*
 * pcmoe.h — C ABI of an MI355X (gfx950) library for the Mixture-of-Experts expert layer of
 * PC-MoE collaborative training (arXiv 2506.02965).
 *
 * The layer is the paper's "expert step": gating (Alg. 7), dispatch of each token to the
 * hosts of its selected experts and the owner-side weighted combine (Alg. 3), the experts'
 * forward and backward passes on their host (Alg. 6), and the gradient hand-back of Alg. 5.
 * One call of this library serves one party's shard of the global expert pool (Sec. 3.1 (2)):
 * the hosted routed experts are the contiguous global ids [local_begin, local_begin+local_count).
 * Each expert is a SwiGLU block  E(h) = W_down (silu(W_gate h) * (W_up h)).
 *
 * Conventions shared by every call
 *   - Every tensor pointer is a DEVICE pointer owned by the caller; the library never frees it.
 *     Tensor pointers must be 16-byte aligned and workspace pointers 256-byte aligned (as any
 *     hipMalloc / torch allocation is); logit_bias only needs 4-byte alignment.
 *   - Every call only validates its arguments and enqueues kernels on `stream`; it never
 *     allocates, frees or synchronises. Results are ready when the stream reaches them.
 *   - Row-major layouts. Weights are [out, in] (so every contraction reads K contiguously from
 *     at least one operand). `dtype` is the storage type of activations and expert weights;
 *     accumulation is fp32. logits, topk_w, dgate, dlogits and dw_router are always fp32.
 *   - Slots: assignment a = t*k + j is token t's j-th selected expert (j = rank by score).
 *   - Row space of the expert buffers (x_perm, y_perm, dy_perm, dx_perm, saved activations):
 *     rows [0, N_loc) hold the hosted routed assignments grouped by expert (N_loc =
 *     offsets[local_count] <= T*k, computed on the device); rows T*k + s*T + t hold shared
 *     expert s applied to token t. The capacity is R = T*k + n_shared*T rows.
 *   - Per-expert counts never travel to the host: grouped kernels read `offsets` on device.
 *   - Errors: a non-zero moe_status is returned and nothing is enqueued; arguments are
 *     checked before any launch. moe_last_error() gives a thread-local explanation.
 *     MOE_ERR_INVALID_ARGUMENT: null or misaligned pointer, k<1, k>E, bad shard range,
 *       local_count < 1 (a party hosts at least one routed expert), bias_groups not dividing T, bad dtype.
 *     MOE_ERR_UNSUPPORTED: d_model or d_ff not a multiple of 128, E > 256, k > 8,
 *       local_count + n_shared > 511, T*k beyond int32 slot indexing, (T + 256) * max(d_model, 2*d_ff) *
 *       elem_bytes >= 2^31 (one expert group's widest operand and a tile past its end, addressed with 32-bit
 *       offsets), or (m + 256) * m * elem_bytes >= 2^31 with m = max(d_model, d_ff) (one expert's weight
 *       matrix and a tile past its end).
 *     MOE_ERR_WORKSPACE_TOO_SMALL: ws_bytes below moe_workspace_size(). MOE_ERR_HIP: a kernel launch failed.
 *   - Calls are reentrant; concurrent calls must use distinct output and workspace buffers.
 *   - Global state: the thread-local error string, and the per-kernel timing state of the measurement
 *     calls at the end of this header (off unless moe_kernel_timing(1) is called; its events are created by
 *     that call, never by a layer call).
 */
#ifndef PCMOE_H
#define PCMOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARGUMENT = 1,
  MOE_ERR_UNSUPPORTED = 2,
  MOE_ERR_WORKSPACE_TOO_SMALL = 3,
  MOE_ERR_HIP = 4
} moe_status;

typedef enum { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype;

/* Shape of one layer call. */
typedef struct {
  int32_t T;            /* tokens in the batch, >= 1 (an empty batch is MOE_ERR_INVALID_ARGUMENT) */
  int32_t d_model;      /* hidden size d */
  int32_t d_ff;         /* expert inner size f */
  int32_t n_experts;    /* E: global routed experts = router width (every party owns the whole
                           gating layer, Sec. 3.1 (3)) */
  int32_t top_k;        /* k selected experts per token (Alg. 7 TopKIndices) */
  int32_t local_begin;  /* first hosted routed expert (global id) */
  int32_t local_count;  /* number of hosted routed experts */
  int32_t n_shared;     /* always-active shared experts, weight 1 (Sec. 3.1 footnote) */
  int32_t renormalize;  /* 1: gate weights renormalised over the k selected experts;
                           0: w = p[I] exactly as Alg. 7 states */
  int32_t dtype;        /* moe_dtype */
} moe_desc;

/* moe_workspace_size(which) selectors */
enum {
  MOE_WS_PERMUTE = 0,     /* scratch of moe_permute */
  MOE_WS_FFN_SAVED = 1,   /* activations saved by moe_expert_ffn_fwd for the backward */
  MOE_WS_FFN_FWD = 2,     /* scratch of moe_expert_ffn_fwd */
  MOE_WS_FFN_BWD = 3,     /* scratch of moe_expert_ffn_bwd */
  MOE_WS_ROUTE_BWD = 4    /* scratch of moe_route_bwd */
};

/* Bytes of device memory the selected buffer needs for this shape (0 if none). */
size_t moe_workspace_size(const moe_desc* desc, int which);

/*
 * Gating, Alg. 7: scores s = W_g h (+ bias), p = softmax(s), I = TopKIndices(p), w = p[I]
 * (renormalised over I when desc->renormalize). Selection is decided on the fp32 scores,
 * which are formed with fp64 accumulation and rounded once; equal scores rank the lower
 * expert index first; slots j are in descending score order.
 *   x          [T, d]   dtype
 *   w_router   [E, d]   dtype
 *   logit_bias [bias_groups, E] fp32 or NULL; token t adds row t / (T / bias_groups)
 *   logits     [T, E]   fp32 out (scores incl. bias)
 *   topk_idx   [T, k]   int32 out (global expert ids)
 *   topk_w     [T, k]   fp32 out
 */
moe_status moe_route(const moe_desc* desc, const void* x, const void* w_router, const float* logit_bias,
                     int32_t bias_groups, float* logits, int32_t* topk_idx, float* topk_w, hipStream_t stream);

/*
 * Dispatch, Alg. 3 (each token's hidden state to the hosts of its selected experts): a stable counting sort of
 * the hosted slots by expert and a gather of their token rows.
 *   topk_idx    [T, k] int32 in
 *   x           [T, d] dtype in
 *   counts      [local_count]   int32 out: rows per hosted expert
 *   offsets     [local_count+1] int32 out: exclusive prefix sums; offsets[local_count] = N_loc
 *   row_to_slot [T*k] int32 out: rows [0, N_loc) give their slot; rows >= N_loc get -1
 *   slot_to_row [T*k] int32 out: the inverse; -1 for slots whose expert is hosted elsewhere
 *   x_perm      [T*k, d] dtype out: rows [0, N_loc) = x[row_to_slot / k]; other rows untouched
 *   ws          MOE_WS_PERMUTE bytes of scratch
 */
moe_status moe_permute(const moe_desc* desc, const int32_t* topk_idx, const void* x, int32_t* counts,
                       int32_t* offsets, int32_t* row_to_slot, int32_t* slot_to_row, void* x_perm,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_permute without a workspace argument, for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc). Same arguments, outputs and errors as
 * moe_permute, bit for bit the same results. Its scratch is a fixed 1 MiB device array inside the library, one
 * per GPU, held until the process ends (looked up on the first call on each device); the call allocates
 * nothing. MOE_ERR_UNSUPPORTED when the shape needs more scratch than that:
 * ceil(T*k / 1024) * local_count * 4 bytes > 1 MiB. Every call on one GPU shares that scratch: calls that overlap
 * in time on the same GPU (concurrent streams, or threads) race and must be serialised by the caller.
 */
moe_status moe_permute_noalloc(const moe_desc* desc, const int32_t* topk_idx, const void* x, int32_t* counts,
                               int32_t* offsets, int32_t* row_to_slot, int32_t* slot_to_row, void* x_perm,
                               hipStream_t stream);

/*
 * ForwardExpert of Alg. 6 for every hosted expert and every shared expert (grouped GEMMs):
 * G = h W_gate^T, U = h W_up^T, H = silu(G) * U, O = H W_down^T.
 *   x       [T, d]  dtype: input rows of the shared experts
 *   x_perm  [T*k, d] dtype: input rows of the routed experts (from moe_permute)
 *   offsets [local_count+1] int32 (from moe_permute)
 *   w_gate  [local_count + n_shared, f, d] dtype (shared experts last)
 *   w_up    [local_count + n_shared, f, d] dtype
 *   w_down  [local_count + n_shared, d, f] dtype
 *   y_perm  [R, d] dtype out (row space above)
 *   saved   MOE_WS_FFN_SAVED bytes out: G, U, H and the grouped-GEMM tile plan for the backward, and the tile
 *           counters of the gate/up and down-projection launches (opaque; calls that overlap on the GPU need their
 *           own)
 *   ws      MOE_WS_FFN_FWD bytes of scratch (currently 0: ws may be NULL)
 */
moe_status moe_expert_ffn_fwd(const moe_desc* desc, const void* x, const void* x_perm, const int32_t* offsets,
                              const void* w_gate, const void* w_up, const void* w_down, void* y_perm,
                              void* saved, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Owner-side combine of Alg. 3: y_t = sum_{j hosted} w_tj * y_perm[slot_to_row[t*k+j]]
 *                                     + sum_s y_perm[T*k + s*T + t]   (fp32 sums, slots j in order).
 *   y [T, d] dtype out. Tokens with no hosted expert and no shared expert get 0.
 */
moe_status moe_combine(const moe_desc* desc, const void* y_perm, const int32_t* slot_to_row, const float* topk_w,
                       void* y, hipStream_t stream);

/*
 * Adjoint of the combine (Alg. 5 and Sec. 3.2 "Backward propagation": the host of an expert
 * receives the gradient w.r.t. that expert's output):
 *   dy_perm[row(t,j)] = w_tj * dy_t           [T*k, d] dtype out (rows >= N_loc untouched)
 *   dgate[t, j]       = <dy_t, y_perm[row(t,j)]>  [T, k] fp32 out, 0 for slots hosted elsewhere
 * Shared experts take dy itself as their output gradient (see moe_expert_ffn_bwd).
 */
moe_status moe_combine_bwd(const moe_desc* desc, const void* dy, const void* y_perm, const int32_t* slot_to_row,
                           const float* topk_w, void* dy_perm, float* dgate, hipStream_t stream);

/*
 * BackwardExpert of Alg. 6 (grouped GEMMs), for hosted and shared experts:
 *   dH = dO W_down, dU = dH * silu(G), dG = dH * U * silu'(G),
 *   dW_down = dO^T H, dW_gate = dG^T h, dW_up = dU^T h, dh = dG W_gate + dU W_up.
 *   dy       [T, d] dtype: output gradient of the shared experts
 *   dy_perm  [T*k, d] dtype: output gradient of the routed rows (from moe_combine_bwd)
 *   saved    from moe_expert_ffn_fwd of the same call shape and inputs
 *   dx_perm  [R, d] dtype out: input gradient per row (row space)
 *   dw_gate, dw_up [local_count + n_shared, f, d] dtype out; dw_down [.., d, f] dtype out.
 *            Hosted experts that received no row get exact zeros.
 *   ws       MOE_WS_FFN_BWD bytes of scratch: dG|dU, and two tile counters that the call zeroes before its
 *            GEMM launches claim their last weight-gradient tiles from them. Calls that overlap on the
 *            GPU need workspaces of their own.
 */
moe_status moe_expert_ffn_bwd(const moe_desc* desc, const void* x, const void* x_perm, const void* dy,
                              const void* dy_perm, const int32_t* offsets, const void* w_gate, const void* w_up,
                              const void* w_down, const void* saved, void* dx_perm, void* dw_gate, void* dw_up,
                              void* dw_down, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Adjoint of Alg. 7's gating on the data owner (Sec. 3.2: the gating network needs the
 * gradient w.r.t. each activated expert's input and gate):
 *   renormalize=1: dlogits[t, I_tj] = w_tj (dgate_tj - sum_j' w_tj' dgate_tj'), 0 elsewhere
 *   renormalize=0: dlogits[t, e] = p_te (g_te - sum_e' p_te' g_te'), g = dgate scattered onto E
 *   dw_router = dlogits^T x   [E, d] fp32 out (deterministic fixed-order reduction over T)
 *   logits [T, E] fp32 in (needed for renormalize=0; may be NULL when renormalize=1)
 *   dlogits [T, E] fp32 out
 *   ws      MOE_WS_ROUTE_BWD bytes of scratch
 * Requires local_count == n_experts (the owner has every slot's dgate).
 */
moe_status moe_route_bwd(const moe_desc* desc, const void* x, const float* logits, const int32_t* topk_idx,
                         const float* topk_w, const float* dgate, float* dlogits, float* dw_router, void* ws,
                         size_t ws_bytes, hipStream_t stream);

/*
 * Hand-back of the input gradient (Sec. 3.2: each host returns one activation-sized gradient
 * to the data owner), summed per token:
 *   dx_t = sum_{j hosted} dx_perm[row(t,j)] + sum_s dx_perm[T*k + s*T + t]
 *          (+ sum_e dlogits[t, e] * w_router[e, :] when dlogits is not NULL)
 *   dx [T, d] dtype out.
 */
moe_status moe_permute_bwd(const moe_desc* desc, const void* dx_perm, const int32_t* slot_to_row,
                           const float* dlogits, const void* w_router, void* dx, hipStream_t stream);

/* Optimiser of the expert update. */
typedef enum { MOE_OPT_SGD = 0, MOE_OPT_ADAMW = 1 } moe_opt_kind;
typedef struct {
  int32_t kind;          /* moe_opt_kind */
  float lr;              /* learning rate, > 0 */
  float beta1, beta2;    /* AdamW moment decays, each in [0, 1) */
  float eps;             /* AdamW denominator term, > 0 */
  float weight_decay;    /* decoupled decay factor, >= 0 (the parameter shrinks by lr * weight_decay) */
  int32_t step;          /* AdamW step number t >= 1 (bias corrections 1 - beta^t) */
} moe_opt;

/*
 * The update of the expert parameters that ends the host's step in Alg. 6 (after BackwardExpert) for every hosted
 * routed expert and every shared expert, elementwise in fp32:
 *   SGD:    p <- p - lr * (g + weight_decay * p)
 *   AdamW:  p <- p * (1 - lr * weight_decay);  m <- beta1 m + (1 - beta1) g;  v <- beta2 v + (1 - beta2) g^2;
 *           p <- p - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 * The paper leaves the optimiser open; AdamW with decoupled weight decay (Loshchilov & Hutter, ICLR 2019)
 * and plain SGD are the two offered.
 *   w_gate, w_up, w_down      the expert weights (layouts of moe_expert_ffn_fwd), dtype, updated in place
 *   dw_gate, dw_up, dw_down   their gradients (from moe_expert_ffn_bwd), dtype
 *   master  NULL or fp32 [P]: the master copy of the parameters. When given, the update starts from it,
 *           it receives the new values and the dtype weights receive their rounding (round to nearest
 *           even); when NULL the update starts from the dtype weights themselves.
 *   m, v    fp32 [P] AdamW moments, updated in place (ignored, may be NULL, for SGD)
 * P = (local_count + n_shared) * 3 * d_ff * d_model; the fp32 arrays hold w_gate, then w_up, then w_down,
 * each in its own layout. The descriptor is checked as for the other calls; the update uses its expert
 * counts, d_model, d_ff and dtype. All pointers 16-byte aligned. Errors as above, and
 * MOE_ERR_INVALID_ARGUMENT for an optimiser setting outside the ranges stated in moe_opt or a NULL m / v
 * under AdamW. Calls that overlap on the same parameters race.
 */
moe_status moe_expert_update(const moe_desc* desc, const moe_opt* opt, void* w_gate, void* w_up, void* w_down,
                             const void* dw_gate, const void* dw_up, const void* dw_down, float* master, float* m,
                             float* v, hipStream_t stream);

/* Per-kernel timing with HIP events recorded around every kernel launch on its own stream
 * (measurement aid; off by default). enable=1 clears the totals and starts recording; its first use creates
 * a pool of 8192 HIP events and a table for 4096 launches, kept until the process ends (MOE_ERR_HIP if the
 * events cannot be created). Layer calls take events from the pool and allocate nothing; launches beyond the
 * pool go unrecorded and are reported as "(unrecorded)". enable=0 stops recording. */
moe_status moe_kernel_timing(int enable);
/* Restricts recording to the launches of one kernel (e.g. "gemm_bwd_dx"); NULL records all. */
moe_status moe_kernel_timing_select(const char* kernel_name);
/* Waits for the recorded events and writes "name count total_ms\n" lines into buf. Returns
 * the number of bytes needed (including the terminating NUL). */
size_t moe_kernel_timing_report(char* buf, size_t buf_bytes);

const char* moe_status_string(moe_status status);
const char* moe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PCMOE_H */
