/*
 * bsa.h - C ABI of the Ball Sparse Attention (BSA) layer library for AMD MI355X (gfx950).
 *
 * The layer (arXiv 2506.12541, Section 2.2) orders an irregular point set with a ball
 * tree, then sums three attention branches over the ordered tokens, each scaled by a
 * sigmoid gate (Eq. 9): attention inside each ball (Ball Tree Attention, Eq. 3),
 * attention to MLP-compressed key/value blocks (Eq. 5), and attention to the top-k key
 * blocks selected per query group from the compressed scores (Eq. 6-8, 10-12).
 *
 * General conventions
 *  - Every pointer argument is a device pointer on the current HIP device unless stated
 *    otherwise. Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL = the default stream) and returns once its kernels are queued.
 *  - bsa_forward and bsa_backward run independent branches concurrently: on first use on
 *    a device the library creates one auxiliary stream (default priority) and two events
 *    for that device and keeps them until the process ends. (The forward of a bf16 layer
 *    without padding, whose ball and compressed attention share one launch, runs on
 *    `stream` alone.) Work on the auxiliary stream
 *    starts after an event recorded on `stream` and is joined back into `stream` before
 *    the call returns, so `stream` alone orders the call against the caller's other work.
 *    Calls from several threads are serialised while they enqueue. bsa_set_streams(1)
 *    runs every branch on `stream` instead (0: also without shared launches).
 *  - The library never allocates device memory and keeps no pointer after a call
 *    returns. The caller owns every buffer; sizes come from bsa_sizes() and
 *    bsa_ball_tree_workspace_bytes().
 *  - Arguments are validated on the host before anything is launched; an invalid call
 *    returns a non-zero status and launches nothing. A failed launch returns
 *    BSA_ERR_HIP. A fault inside a kernel surfaces at the caller's next synchronisation.
 *    bsa_last_error() gives a human-readable detail of the last failure on the calling
 *    thread. No C++ exception crosses this boundary.
 *  - Token layout: Q, K, V, O and their gradients are [B, H, N, d] row-major in ball
 *    order (slot order of the tree), so a ball, a compression block, a selection block
 *    and a query group of one head are each one contiguous run of rows.
 */
#ifndef BSA_H
#define BSA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BSA_OK = 0,
  BSA_ERR_INVALID_ARGUMENT = 1,   /* a size, pointer or parameter is invalid            */
  BSA_ERR_UNSUPPORTED = 2,        /* valid but not implemented (e.g. head_dim not 32/64) */
  BSA_ERR_WORKSPACE_TOO_SMALL = 3,
  BSA_ERR_HIP = 4                 /* a HIP runtime call or kernel launch failed          */
} bsa_status_t;

typedef enum { BSA_F32 = 0, BSA_BF16 = 1 } bsa_dtype_t;
typedef enum { BSA_POOL_MLP = 0, BSA_POOL_MEAN = 1 } bsa_pool_t;
/* Coarse queries of the selection scores: the group mean of Eq. 11, or an MLP phi_q of
 * each block of l queries (Eq. 13). */
typedef enum { BSA_QC_MEAN = 0, BSA_QC_MLP = 1 } bsa_qcoarsen_t;

/* Layer hyper-parameters (notation of Section 2). */
typedef struct {
  int32_t batch;          /* B: independent point clouds                               */
  int32_t n;              /* N: token slots per cloud (power of two, >= 64)            */
  int32_t heads;          /* H                                                         */
  int32_t head_dim;       /* d: 32 or 64                                               */
  int32_t ball_size;      /* m: ball size of Eq. 3 (power of two, divides N)           */
  int32_t cmp_block;      /* l: compression block length of Eq. 5 (power of two)       */
  int32_t cmp_stride;     /* compression stride; must equal cmp_block (Eq. 5)          */
  int32_t slc_block;      /* l': selection block length of Eq. 8 (l'=r*l, r in 1,2,4;
                             multiple of 16; divides m)                                */
  int32_t topk;           /* k*: selected blocks per group (Eq. 7), 1..16; also
                             (16/g or 1) * k* * l' <= 4096                             */
  int32_t group_size;     /* g: query group size of Eq. 10: 1 (per-token selection, bf16
                             only) or a power of two >= 8 dividing m                   */
  int32_t mask_own_ball;  /* 1: a group may not select blocks of its own ball          */
  int32_t store_lse;      /* 1: the forward keeps each branch's log-sum-exp rows for the
                             backward; 0: they are not kept (saved.lse is NULL) and the
                             backward recomputes them by the branches' forward kernels
                             without the value products (same tiles and order: equal
                             to the stored rows bit for bit)                          */
  int32_t deterministic;  /* 0 or 1, no effect: every kernel is deterministic (no float
                             atomics; fixed-order sums), so both values give
                             bit-identical results                                     */
  int32_t kv_pool;        /* bsa_pool_t: MLP (default) or mean pooling of Eq. 5        */
  int32_t dtype;          /* bsa_dtype_t of Q, K, V, O, dO and the saved branch outputs */
  float softmax_scale;    /* 0 -> 1/sqrt(d)                                            */
  int32_t q_coarsen;      /* bsa_qcoarsen_t: BSA_QC_MEAN (default) or BSA_QC_MLP (Eq. 13-14;
                             needs group_size == cmp_block)                            */
  int32_t group_compression; /* 1: the compression branch attends from the coarse queries
                             and copies each result to the real queries of its block
                             (Eq. 15; needs group_size == cmp_block and n/cmp_block >= 64) */
} bsa_params_t;

/* One compression MLP phi (Eq. 5; also phi_q of Eq. 13): y = GELU_erf(x W1 + b1) W2 + b2
 * for the token-major flatten x of an l x d block (dummy rows zero). Float32, shared
 * across heads:
 * w1 [l*d, d], b1 [d], w2 [d, d], b2 [d], row-major. For bf16 layers w1 should hold
 * bf16-representable values: the first layer runs on bf16 matrix cores. */
typedef struct { const float *w1, *b1, *w2, *b2; } bsa_mlp_t;
typedef struct { float *w1, *b1, *w2, *b2; } bsa_mlp_grad_t;

/* Tensors the forward pass saves for the backward pass (all device, caller-owned).
 * bsa_saved_view() carves them out of one buffer of bsa_sizes()'s saved_bytes. */
typedef struct {
  int32_t* sel_idx;  /* [B, H, N/g, k*] selected block ids, ascending, -1 = empty slot  */
  float* lse;        /* [3, B, H, N] natural-log log-sum-exp per branch, -inf = no key;
                        NULL with store_lse = 0 (if set anyway, the forward fills it and
                        the backward still recomputes the rows)                         */
  void* o_branch;    /* [2, B, H, N, d] dtype: ball (0) and selection (1) outputs       */
  float* kcmp;       /* [B, H, N/l, d] compressed keys                                  */
  float* vcmp;       /* [B, H, N/l, d] compressed values                                */
  float* hid_k;      /* [B, H, N/l, d] hidden pre-activation of phi_k                   */
  float* hid_v;      /* [B, H, N/l, d] hidden pre-activation of phi_v                   */
  uint8_t* cvalid;   /* [B, N/l] 1 if the compression block holds a real token          */
  float* qcmp;       /* [B, H, N/g, d] coarse queries of the selection (Eq. 11 or 13)   */
  float* hid_q;      /* [B, H, N/l, d] hidden pre-activation of phi_q (BSA_QC_MLP)      */
  float* ocmp;       /* [B, H, N/l, d] coarse attention outputs of group compression    */
  float* o_cmp;      /* [B, H, N, d] float32 output of the compression branch. Kept
                        unrounded: the backward's softmax delta rowsum(dO o) comes from
                        it, and an error in that delta is common to every compressed key
                        of the query, so it would add up over the blocks in the
                        compression MLP's weight gradients                              */
} bsa_saved_t;

/* ---- Ball tree (Section 2.1 "Ball Tree Attention"; the ordering every branch uses) ---- */

/* Workspace bytes for bsa_build_ball_tree with these sizes (0 on invalid sizes). */
size_t bsa_ball_tree_workspace_bytes(int64_t n_real, int64_t n_pad, int32_t dim, int32_t batch);

/* Order each cloud by recursive median splits: a node of capacity C (a power of two)
 * holding the point set S splits on the axis of largest spread (max - min, formed in
 * float64; equal spreads -> lowest axis), its points ordered by (coordinate, index)
 * with -0.0 equal to +0.0; the first ceil(|S|/2) go to the left child (slots
 * [0, C/2)), the rest to the right child; recursion down to single slots.
 *   points: [batch, n_real, dim] float32, finite; dim = 3 (2 and 1 also accepted).
 *   perm:   [batch, n_pad] int32 output; slot -> point index within its cloud, -1 for a
 *           padding slot. 1 <= n_real <= n_pad, n_pad a power of two, n_pad <= 2^24.
 *   ws:     workspace of at least bsa_ball_tree_workspace_bytes() bytes. */
bsa_status_t bsa_build_ball_tree(const float* points, int64_t n_real, int32_t dim,
                                 int64_t n_pad, int32_t batch, int32_t* perm,
                                 void* ws, size_t ws_bytes, void* stream);

/* bsa_build_ball_tree without a workspace argument and without any device allocation, for
 * callers that cannot allocate (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, ordering and errors as
 * bsa_build_ball_tree, minus ws / ws_bytes. The workspace is a static device array of the
 * library (10.7 MB on each device the library runs on, held until the process
 * ends) that covers batch * n_pad <= 131072 slots; larger sizes return
 * BSA_ERR_UNSUPPORTED and launch nothing. Every call on one device shares that array and
 * overwrites it: calls that overlap in time on one device (e.g. on two streams without
 * ordering between them) race and give wrong orderings; calls ordered on one stream are
 * safe. Nothing in the array needs clearing between calls (every word is written before
 * it is read). */
bsa_status_t bsa_build_ball_tree_noalloc(const float* points, int64_t n_real, int32_t dim, int64_t n_pad,
                                         int32_t batch, int32_t* perm, void* stream);

/* Gather per-point rows into ball order (the ordering step before Eq. 3):
 *   src  [batch, n_real, heads*head_dim] (dtype) -> dst [batch, heads, n_pad, head_dim],
 *   dst row = 0 where perm is -1. valid_out [batch, n_pad] (may be NULL) receives
 *   1 for real slots and 0 for padding. head_dim may be any value >= 1 (e.g. heads=1,
 *   head_dim=3 orders the gate logits). */
bsa_status_t bsa_permute(const void* src, const int32_t* perm, int64_t n_real, int64_t n_pad,
                         int32_t batch, int32_t heads, int32_t head_dim, int32_t dtype,
                         void* dst, uint8_t* valid_out, void* stream);

/* Inverse of bsa_permute: src [batch, heads, n_pad, head_dim] -> dst [batch, n_real,
 * heads*head_dim]; padding slots are dropped. dtype BSA_F32 or BSA_BF16. */
bsa_status_t bsa_unpermute(const void* src, const int32_t* perm, int64_t n_real, int64_t n_pad,
                           int32_t batch, int32_t heads, int32_t head_dim, int32_t dtype,
                           void* dst, void* stream);

/* ---- The layer (Section 2.2, Eq. 3, 5-12, 9) ---- */

/* Validate p and report the sizes of the forward workspace, the backward workspace and
 * the saved-tensor buffer. Any pointer may be NULL. */
bsa_status_t bsa_sizes(const bsa_params_t* p, size_t* ws_fwd_bytes, size_t* ws_bwd_bytes,
                       size_t* saved_bytes);

/* Point the fields of *out into the caller's buffer `base` of saved_bytes bytes
 * (256-byte aligned sub-buffers). Host-only arithmetic; launches nothing. */
bsa_status_t bsa_saved_view(const bsa_params_t* p, void* base, bsa_saved_t* out);

/* Forward pass.
 *   q, k, v: [B, H, N, d] dtype in ball order. valid: [B, N] uint8 (1 = real token) or
 *   NULL (all real). gate: [B, N, 3] float32 logits gamma_b in branch order (ball,
 *   compression, selection), shared across heads (Eq. 9). phi_k / phi_v: compression
 *   MLPs for keys / values (ignored for BSA_POOL_MEAN). phi_q: the query-coarsening MLP
 *   (read only for BSA_QC_MLP; may be NULL otherwise).
 *   o: [B, H, N, d] dtype output = sum_b sigmoid(gamma_b) * o_b; rows of padding slots 0.
 *   saved: filled for bsa_backward (and readable as per-branch outputs, LSE and the
 *   selected block ids). ws: at least ws_fwd_bytes. */
bsa_status_t bsa_forward(const bsa_params_t* p, const void* q, const void* k, const void* v,
                         const uint8_t* valid, const float* gate, const bsa_mlp_t* phi_k,
                         const bsa_mlp_t* phi_v, const bsa_mlp_t* phi_q, void* o,
                         const bsa_saved_t* saved, void* ws, size_t ws_bytes, void* stream);

/* Backward pass of bsa_forward given dO = d(loss)/d(o) ([B, H, N, d] dtype).
 * Outputs (overwritten, float32): dq, dk, dv [B, H, N, d]; dgate [B, N, 3];
 * dphi_k / dphi_v weight gradients summed over batch, heads and blocks (may be NULL for
 * BSA_POOL_MEAN). dphi_q: gradient of phi_q, which receives one only through group
 * compression (required for BSA_QC_MLP with group_compression = 1, else may be NULL and
 * is not written). No gradient flows through the top-k selection. Rows of padding slots
 * get zero gradients. ws: at least ws_bwd_bytes. */
bsa_status_t bsa_backward(const bsa_params_t* p, const void* q, const void* k, const void* v,
                          const uint8_t* valid, const float* gate, const bsa_mlp_t* phi_k,
                          const bsa_mlp_t* phi_v, const bsa_mlp_t* phi_q, const bsa_saved_t* saved,
                          const void* d_o, float* dq, float* dk, float* dv, float* dgate,
                          const bsa_mlp_grad_t* dphi_k, const bsa_mlp_grad_t* dphi_v,
                          const bsa_mlp_grad_t* dphi_q, void* ws, size_t ws_bytes, void* stream);

/* Streams used by bsa_forward and bsa_backward: 2 (default) = the caller's stream plus
 * the auxiliary stream (in the forward only where ball and compressed attention run as
 * separate launches), 1 = the caller's stream only (branches run one after another,
 * e.g. to time each alone), 0 = as 1, and the branches that otherwise share a launch
 * (ball and compressed attention forward, and their key-major backward passes, for bf16
 * layers without padding) get launches of their own, so that each branch can be timed.
 * Results are the same bit for bit in every mode. Process-wide; BSA_ERR_INVALID_ARGUMENT
 * for other values. */
bsa_status_t bsa_set_streams(int32_t n);

/* ---- The transformer block around the layer (Section 3.1) ----
 *
 * The paper's model stacks 18 blocks of RMSNorm, a BSA layer and a SwiGLU. One block, with
 * C = heads * head_dim channels and F SwiGLU hidden units, on tokens x [B, N, C] float32 in
 * ball order (padding rows zero):
 *   h = x + merge(BSA(Q, K, V; gate)) W_o^T,   [Q | K | V] = RMSNorm_1(x) W_qkv^T,
 *   gate = RMSNorm_1(x) W_g^T,   y = h + (silu(z W_1^T) * (z W_3^T)) W_2^T, z = RMSNorm_2(h),
 * RMSNorm(t) = t / sqrt(mean(t^2) + 1e-6) * gain; maps are bias-free and stored [out, in]
 * (head h of Q takes output columns h d .. h d + d - 1 of W_qkv, then K, then V).
 * Precision: bf16 layers only. The channel products take bf16 operands (round to nearest
 * even) and accumulate in float32; Q, K, V, the layer output, u = z W_1^T, w = z W_3^T
 * and silu(u) w are stored in bf16; the residual stream, the norms and the gate logits
 * (from the unrounded norm output and float32 W_g) are float32. In the backward pass the
 * gradients entering a product (dy, du, dw, dh, dO, dQ/dK/dV) are rounded to bf16.
 * Requirements beyond bsa_sizes: dtype BSA_BF16, C in {128, 256, 512, 1024}, F a positive
 * multiple of 128 (BSA_ERR_UNSUPPORTED otherwise). */
typedef struct {
  const float *g1;      /* [C]     gain of RMSNorm_1                                    */
  const float *wqkv;    /* [3C, C]                                                      */
  const float *wg;      /* [3, C]  gate logits (ball, compression, selection)           */
  const float *wo;      /* [C, C]                                                       */
  const float *g2;      /* [C]     gain of RMSNorm_2                                    */
  const float *w1, *w3; /* [F, C]                                                       */
  const float *w2;      /* [C, F]                                                       */
  bsa_mlp_t phi_k, phi_v, phi_q;  /* the layer's MLPs (phi_q read only for BSA_QC_MLP)  */
} bsa_block_weights_t;

/* Gradients of the weights (float32, same shapes, overwritten). phi_q: written only for
 * BSA_QC_MLP with group compression (as in bsa_backward). */
typedef struct {
  float *g1, *wqkv, *wg, *wo, *g2, *w1, *w3, *w2;
  bsa_mlp_grad_t phi_k, phi_v, phi_q;
} bsa_block_grads_t;

/* Tensors the block's forward pass saves for its backward pass (device, caller-owned;
 * bsa_block_saved_view() carves them out of one buffer). M = B * N token rows. */
typedef struct {
  bsa_saved_t layer;    /* the layer's own saved tensors                               */
  float* rstd1;         /* [M]        1 / rms of each row of x                          */
  float* rstd2;         /* [M]        1 / rms of each row of h                          */
  void* xn1;            /* [M, C]     bf16 RMSNorm_1(x)                                 */
  float* gate;          /* [B, N, 3]  gate logits                                       */
  void* q;              /* [B, H, N, d] bf16 (k, v likewise)                            */
  void* k;
  void* v;
  void* o;              /* [B, H, N, d] bf16 layer output                               */
  float* h;             /* [M, C]     residual stream after the attention sublayer      */
  void* xn2;            /* [M, C]     bf16 RMSNorm_2(h)                                 */
  void* uw;             /* [M, 2F]    bf16 u (columns 0..F-1) and w (F..2F-1)           */
  void* a;              /* [M, F]     bf16 silu(u) w                                    */
} bsa_block_saved_t;

/* Validate and report the forward workspace, backward workspace and saved-buffer sizes of
 * one block with F = ffn_dim. Any size pointer may be NULL. */
bsa_status_t bsa_block_sizes(const bsa_params_t* p, int32_t ffn_dim, size_t* ws_fwd_bytes,
                             size_t* ws_bwd_bytes, size_t* saved_bytes);

/* Point the fields of *out into `base` (saved_bytes of bsa_block_sizes). Host-only. */
bsa_status_t bsa_block_saved_view(const bsa_params_t* p, int32_t ffn_dim, void* base,
                                  bsa_block_saved_t* out);

/* Block forward: x [B, N, C] float32 -> y [B, N, C] float32 (y may not alias x). valid as
 * in bsa_forward. ws: at least ws_fwd_bytes. Asynchronous on `stream` (the layer inside
 * may also use the library's auxiliary stream, joined before return). */
bsa_status_t bsa_block_forward(const bsa_params_t* p, int32_t ffn_dim, const bsa_block_weights_t* w,
                               const float* x, const uint8_t* valid, float* y,
                               const bsa_block_saved_t* saved, void* ws, size_t ws_bytes, void* stream);

/* Block backward given dy = d(loss)/d(y) [B, N, C] float32: dx [B, N, C] float32 and the
 * weight gradients (summed over tokens in a fixed order; no float atomics). x and saved as
 * given to / filled by bsa_block_forward. ws: at least ws_bwd_bytes. */
bsa_status_t bsa_block_backward(const bsa_params_t* p, int32_t ffn_dim, const bsa_block_weights_t* w,
                                const float* x, const uint8_t* valid, const bsa_block_saved_t* saved,
                                const float* dy, float* dx, const bsa_block_grads_t* dw, void* ws,
                                size_t ws_bytes, void* stream);

/* ---- Measurement support (not part of the layer's computation) ---- */

/* on = 1: start recording, clearing earlier records; on = 0: stop and clear. While on,
 * every timed phase of the library records a start and a stop HIP event on the stream
 * its kernels are launched on (phases on the two streams of a call may overlap in time). Phases: "tree", "permute", "fwd.compress", "fwd.select",
 * "fwd.ball", "fwd.cmp", "fwd.slc", "fwd.gate", "bwd.lse" (store_lse = 0), "bwd.gate", "bwd.dq_ball", "bwd.dq_cmp",
 * "bwd.dq_slc", "bwd.kv_ball", "bwd.kv_cmp", "bwd.mlp", "bwd.slc_csr", "bwd.slc_kv", and
 * for the block "blk.norm", "blk.gemm" (activation products), "blk.wgrad" (weight
 * gradients), "blk.elem" (SwiGLU, casts, layout changes).
 * Host-side bookkeeping only; no device memory is allocated. */
bsa_status_t bsa_timing_enable(int32_t on);

/* Restrict the recording to the comma-separated phase names in `phases` (NULL or "" =
 * every phase), so that a measured region carries the events of the phases it reports
 * and no others. Host-side bookkeeping only. */
bsa_status_t bsa_timing_select(const char* phases);

/* Sum of the recorded durations of `phase` (milliseconds) and the number of records;
 * waits for the recorded events to complete. */
bsa_status_t bsa_timing_query(const char* phase, double* total_ms, int32_t* count);

const char* bsa_status_string(bsa_status_t s);
/* Detail of the last failure on the calling thread ("" if none). */
const char* bsa_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* BSA_H */
