/*
 * clearmoe.h -- C ABI of the CLEAR-MoE FFN forward on MI355X (gfx950).
 *
 * The layer (arxiv 2606.28516, Eq. 2 and Algorithm 3):
 *     z     = GELU(x W1^T + b1)                       shared fc1, all tokens
 *     h_sh  = (z Vt^T) US^T + b2                      shared SVD basis of fc2,
 *                                                     US = U_r diag(S_r), Vt = V_r^T
 *     a     = top-k of the linear router x Wg^T + bg  (k = 1: Algorithm 3's argmax)
 *     h_res = sum_j gate_j (z Q_{a_j}^T) P_{a_j}^T    per-expert residual, rank q
 *     y     = h_sh + h_res
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is a DEVICE pointer owned by the caller, and the
 *     library keeps none after a call returns.  No entry point allocates
 *     device memory; scratch comes from the caller's workspace.  Host-side
 *     resources that an entry point creates on first use and keeps until
 *     the process ends: clearmoe_ffn_forward_padded, a pinned 256-byte host
 *     buffer per calling thread (and an event per call, destroyed before it
 *     returns); clearmoe_ffn_forward and _ex on a top-2 layer in expert-pair
 *     order, or with class tokens, a side stream and two events per device
 *     (clearmoe_ffn_forward_noalloc creates none); the stage timer, the
 *     events it is started with.
 *   - Matrices are row-major and contiguous.  Weights are stored [out, in]
 *     (the nn.Linear convention), so every product is A[M,K] B[N,K]^T.
 *   - x, W1, US, Vt, P, Q, Wg, ye and y have element type shape->dtype
 *     (CLEARMOE_F32 = float, CLEARMOE_BF16 = bfloat16 bits).  Biases and gates
 *     are always float32; index arrays are int32.  A NULL bias means zero.
 *   - Scratch memory comes from the caller's workspace `ws` of `ws_bytes`
 *     bytes, at least clearmoe_workspace_bytes(shape), 256-byte aligned.
 *   - All work is enqueued on `stream`; nothing is synchronised and nothing is
 *     copied to the host.  The call returns once the kernels are enqueued.
 *   - Arguments are checked on the host before anything is launched: shapes
 *     (T >= 0; D, H >= 1; 1 <= k <= E <= 64; 0 <= r, q <= min(D, H);
 *     T*k < 2^31; D, H, r, q multiples of 8 for bf16 and of 4 for float32),
 *     required pointers non-NULL and 16-byte aligned, the workspace large
 *     enough.  A failed check returns its status and has no side effect.  A
 *     launch failure returns CLEARMOE_ERR_HIP (hipGetLastError).
 *   - The layer entry points clearmoe_ffn_forward, clearmoe_ffn_forward_ex
 *     and clearmoe_dense_ffn_forward also take D, H, r, q that are not such
 *     multiples: those shapes run on zero-padded copies of the operands in
 *     the workspace (clearmoe_workspace_bytes counts them), with the same
 *     routing and y as unpadded (padding adds only zero products, and an
 *     extra hidden unit's activation is GELU(0) = 0); their pointers need
 *     only element alignment (the router's Wg stays 16-byte aligned when it
 *     is an MLP router's [E, hidden] output layer).  clearmoe_route and
 *     clearmoe_route_ex take any D the same way (padded copies of x and the
 *     router's D-wide matrix, counted by clearmoe_workspace_bytes);
 *     clearmoe_dispatch (with rows) and clearmoe_combine take any D
 *     directly, copying and combining rows one element at a time (same
 *     results; their row pointers need element alignment only).  The padded
 *     backend and the stack keep the multiples.
 *   - No C++ exception crosses this interface.  Calls on one stream are
 *     ordered; calls that share a workspace must not overlap in time.
 */
#ifndef CLEARMOE_H
#define CLEARMOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CLEARMOE_OK = 0,
    CLEARMOE_ERR_INVALID_ARG = 1,   /* bad shape, NULL or misaligned pointer */
    CLEARMOE_ERR_UNSUPPORTED = 2,   /* valid but not handled (e.g. dtype) */
    CLEARMOE_ERR_WORKSPACE = 3,     /* ws NULL or smaller than required */
    CLEARMOE_ERR_HIP = 4,           /* a kernel launch failed */
    CLEARMOE_ERR_TOO_LARGE = 5      /* clearmoe_ffn_forward_noalloc: the shape
                                       needs more than its fixed scratch */
} clearmoe_status;

typedef enum { CLEARMOE_F32 = 0, CLEARMOE_BF16 = 1 } clearmoe_dtype;

/* Layer shape.  T tokens, D model width, H fc1 width (d_ffn), E experts,
 * k experts per token, r shared SVD rank, q residual rank per expert.
 * renorm selects the gates of the chosen experts (Sec. III Phase 4 treats
 * the router's scores as a distribution over the E experts; the paper does
 * not say whether the top-k gates are renormalised):
 *   1  the softmax of the k selected logits, renormalised over them (k = 1:
 *      gate 1) -- the reading the benchmark workloads use;
 *   0  the selected experts' probabilities under the softmax over all E
 *      logits (they sum to less than 1 unless k = E).
 * Any other value is rejected (CLEARMOE_ERR_INVALID_ARG); a zero-filled
 * struct therefore asks for the unrenormalised gates. */
typedef struct {
    int32_t T, D, H, E, k, r, q;
    int32_t dtype;                 /* clearmoe_dtype */
    int32_t renorm;                /* 1: renormalised top-k gates; 0: full-softmax gates */
} clearmoe_shape;

/* Flags of clearmoe_dispatch. */
#define CLEARMOE_DISPATCH_HIST_IN_WS 1u  /* ws already holds the per-tile expert
                                            histogram of idx, as left there by
                                            clearmoe_route with the same shape */

/* Library version, (major << 16) | minor. */
int clearmoe_version(void);

/* First 16 hex digits of the SHA-256 of the sources the library was built
 * from (static string, never NULL): lets a caller refuse a stale binary. */
const char* clearmoe_source_digest(void);

/* Human-readable name of a status code (static string, never NULL). */
const char* clearmoe_status_string(int status);

/* Bytes of workspace clearmoe_ffn_forward needs for this shape (enough for
 * every entry point but clearmoe_ffn_forward_padded); 0 if the shape is
 * invalid. */
size_t clearmoe_workspace_bytes(const clearmoe_shape* shape);

/* Router and top-k (Sec. III Phase 4 linear router, with the bias counted in
 * Table C5; Algorithm 3 "a <- argmax(g(x))"; top-k with softmax gates,
 * renormalised over the selected experts unless shape->renorm is 0).
 *   x   [T, D], Wg [E, D] (dtype); bg [E] float32 or NULL.
 *   idx [T, k] int32 out: experts by logit descending, ties to the lower
 *       index; slot 0 is the best.
 *   gate [T, k] float32 out: renorm 1: softmax over the k selected logits
 *       (1.0 at k=1); renorm 0: the selected experts' probabilities under
 *       the softmax over all E logits.
 * The choice is exact: logits are accumulated in float32 by MFMA together
 * with a rigorous bound on their rounding error, and every token whose top-k
 * gaps do not clear that bound is recomputed in double (so ties are decided
 * by the index rule on exact sums).  Gates come from the same logits.
 * ws (required) receives the per-tile expert histogram of the result, which a
 * following clearmoe_dispatch with CLEARMOE_DISPATCH_HIST_IN_WS and the same
 * T, E, k reuses instead of recounting.  Uses shape fields T, D, E, k,
 * dtype, renorm. */
int clearmoe_route(const clearmoe_shape* shape, const void* x, const void* Wg, const float* bg,
                   int32_t* idx, float* gate, void* ws, size_t ws_bytes, hipStream_t stream);

/* Router of a layer.  Sec. III Phase 4 fits one of three routers to the
 * cluster labels (Table C5 compares them): Linear, MLP (one hidden layer,
 * width d/6 there) and Adaptive (top-1, escalated to top-2 when the router is
 * not confident).  Here the scoring function and the selection rule are
 * independent fields, so an MLP router can also select adaptively.
 *   Scores:   hidden == 0: l = x Wg^T + bg, Wg [E, D] (as clearmoe_route);
 *             hidden  > 0: hr = GELU(x Wh^T + bh) rounded once to dtype,
 *             l = hr Wg^T + bg, Wh [hidden, D], Wg [E, hidden].
 *   Choice:   adaptive == 0: the top k = shape->k, gates as clearmoe_route;
 *             adaptive == 1 (shape->k must be 2, E >= 2): the confidence of a
 *             token is its largest softmax probability over all E experts,
 *             p = 1 / sum_e exp(l_e - l_max); p >= tau keeps it at top-1
 *             (idx = (best, -1), gate = (1, 0): slot 1 is empty), otherwise
 *             it takes the top 2 with their softmax renormalised (with
 *             shape->renorm 0: gates (p, 0), or the two probabilities).
 *   Class tokens (Table C6 excludes the class token of each image from
 *   expert dispatch and runs it on the dense path): with dense_stride s > 0
 *   every token t with t % s == 0 gets no expert (all k slots -1, gate 0);
 *   clearmoe_ffn_forward_ex gives it the unexpertised FFN's output,
 *   GELU(x W1^T + b1) W2^T + b2.
 * Weights have element type shape->dtype, biases are float32 (NULL = zero). */
typedef struct {
    const void* Wg;        /* output layer [E, D] (linear) or [E, hidden] (MLP) */
    const float* bg;       /* [E] or NULL */
    const void* Wh;        /* MLP hidden layer [hidden, D]; ignored if hidden == 0 */
    const float* bh;       /* MLP hidden bias [hidden] or NULL */
    const void* W2;        /* dense fc2 [D, H] of the class tokens' path; NULL
                              when dense_stride == 0 (unused by route_ex) */
    int32_t hidden;        /* 0 = linear router; 1..256 = MLP hidden width */
    int32_t adaptive;      /* 0 = top-k; 1 = adaptive top-1 / top-2 */
    int32_t dense_stride;  /* s > 0: token t with t % s == 0 is a class token */
    int32_t reserved;      /* must be 0 */
    double tau;            /* adaptive confidence threshold (any finite value) */
} clearmoe_router;

/* Routing by any router (see clearmoe_router), same outputs and workspace
 * contract as clearmoe_route: idx [T, k] (-1 marks an adaptive router's empty
 * slot), gate [T, k], and the per-tile histogram left in ws for a following
 * clearmoe_dispatch with CLEARMOE_DISPATCH_HIST_IN_WS.  Decisions:
 *   linear: certified as in clearmoe_route; for adaptive selection a token
 *     whose confidence is within the float32 rounding bound of tau is also
 *     recomputed in double, so the threshold is applied to exact logits;
 *   MLP: both layers run in double (products of stored values are exact),
 *     GELU uses the double erf and the hidden values are rounded to dtype
 *     from double in one step; the choice matches exact arithmetic except
 *     where a hidden value lies within double rounding of a dtype rounding
 *     boundary or a top-k gap / |log p - log tau| is below double rounding.
 * Returns CLEARMOE_ERR_INVALID_ARG for a NULL router, hidden outside
 * [0, 256], adaptive not 0 or 1, adaptive with k != 2 or E < 2, a NaN tau,
 * a negative dense_stride, reserved != 0, or NULL / misaligned weights (Wg,
 * Wh, W2 16-byte aligned; biases 4-byte; W2 required by
 * clearmoe_ffn_forward_ex when dense_stride > 0). */
int clearmoe_route_ex(const clearmoe_shape* shape, const clearmoe_router* router, const void* x,
                      int32_t* idx, float* gate, void* ws, size_t ws_bytes, hipStream_t stream);

/* Dispatch: expert histogram, exclusive scan and stable permutation (Sec. III
 * "Dispatch Backends", Grouped: tokens sorted by expert into contiguous
 * sub-batches; Algorithm 3 sort step).
 *   idx     [T, k] int32 in, every entry in [0, E) or -1 (an empty slot, as
 *           an adaptive router leaves it).
 *   counts  [E] out; offsets [E+1] out, offsets[0] = 0, offsets[E] = number
 *           of entries that are not -1 (T*k when there are none).
 *   perm    [T*k] out: perm[p] = a = t*k + j, the assignments of expert 0 in
 *           ascending a, then expert 1, ..., then -1 for p >= offsets[E].
 *   inv     [T*k] out: inv[perm[p]] = p; inv[a] = -1 for an empty slot.
 *   x [T, D] and xperm [T*k, D] (dtype): if both non-NULL, xperm[p] = x[perm[p]/k]
 *           for p < offsets[E] (rows after that are not written).
 * An index outside [-1, E) is not detected on the device; it is the caller's
 * contract (the routers only produce valid ones); such an entry is treated
 * as empty.  Uses T, D, E, k, dtype. */
int clearmoe_dispatch(const clearmoe_shape* shape, const int32_t* idx, void* ws, size_t ws_bytes,
                      int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* inv,
                      const void* x, void* xperm, unsigned flags, hipStream_t stream);

/* Inverse-permute combine (Algorithm 3 "unshuffle h_res; y <- h_sh + h_res",
 * weighted by the gates):  y[t] = sum_j gate[t, j] * ye[inv[t*k + j]],
 * accumulated in float32 in slot order, stored in dtype.
 *   ye [T*k, D] (dtype, expert order), inv [T*k] (-1: empty slot, adds
 *   nothing), gate [T, k], y [T, D] out.
 * Uses T, D, k, dtype. */
int clearmoe_combine(const clearmoe_shape* shape, const void* ye, const int32_t* inv,
                     const float* gate, void* y, hipStream_t stream);

/* The whole layer (Eq. 2, Algorithm 3), all steps on the device.
 *   x [T, D]; W1 [H, D], b1 [H]; US [D, r]; Vt [r, H]; b2 [D];
 *   P [E, D, q], Q [E, q, H] (expert e's residual is P[e] Q[e]);
 *   Wg [E, D], bg [E];  y [T, D] out.
 *   idx_out [T, k] / gate_out [T, k]: optional copies of the routing (NULL ok).
 * bfloat16 mode accumulates in float32; the hidden activation z and the
 * rank-r / rank-q projections are rounded to bfloat16 between products.
 * For k = 1 the shared basis and the residual run as two products over the
 * expert order ([t|u] = z[perm] [Vt;Q_e]^T, then y[perm] = [t|u] [US|P_e]^T
 * + b2); for k > 1 h_sh and h_res are formed apart and combined. */
int clearmoe_ffn_forward(const clearmoe_shape* shape, const void* x, const void* W1,
                         const float* b1, const void* US, const void* Vt, const float* b2,
                         const void* P, const void* Q, const void* Wg, const float* bg, void* y,
                         int32_t* idx_out, float* gate_out, void* ws, size_t ws_bytes,
                         hipStream_t stream);

/* Scratch held by the library for clearmoe_ffn_forward_noalloc, per device. */
#define CLEARMOE_NOALLOC_SCRATCH_BYTES (64u << 20)

/* clearmoe_ffn_forward without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments (minus ws / ws_bytes),
 * kernels and results as clearmoe_ffn_forward; it calls no hipMalloc, hipFree
 * or allocating routine.  Scratch comes from one fixed device array of
 * CLEARMOE_NOALLOC_SCRATCH_BYTES (64 MiB) that the library holds on each
 * device it runs on until the process ends; its address is looked up once per
 * device, on the first call with that device current.  Only the regions the
 * layer's path touches are placed there, packed: every top-1 bfloat16 layer
 * the fused kernel takes needs well under 1 MiB plus its small-batch split
 * partials; the GEMM chains also hold z [T, H] and the low-rank
 * intermediates.  A shape that needs more than the array returns
 * CLEARMOE_ERR_TOO_LARGE before anything is launched.  Every call on a device
 * shares that device's array and leaves its contents behind (the counters it
 * needs are cleared by the call's own fill kernels): calls that overlap in
 * time on one device -- on different streams or threads -- race and must
 * not be issued. */
int clearmoe_ffn_forward_noalloc(const clearmoe_shape* shape, const void* x, const void* W1,
                                 const float* b1, const void* US, const void* Vt, const float* b2,
                                 const void* P, const void* Q, const void* Wg, const float* bg,
                                 void* y, int32_t* idx_out, float* gate_out, hipStream_t stream);

/* The whole layer with any router (see clearmoe_router and
 * clearmoe_route_ex); the other arguments, layouts, results and workspace are
 * those of clearmoe_ffn_forward.  Router weights replace Wg / bg.  An empty
 * slot (adaptive top-1) adds no residual: y = h_sh + h_res of the chosen
 * expert with gate 1.  A class token (dense_stride) gets
 * y = GELU(x W1^T + b1) W2^T + b2 instead, from two extra products over the
 * ceil(T / dense_stride) class rows. */
int clearmoe_ffn_forward_ex(const clearmoe_shape* shape, const clearmoe_router* router,
                            const void* x, const void* W1, const float* b1, const void* US,
                            const void* Vt, const float* b2, const void* P, const void* Q,
                            void* y, int32_t* idx_out, float* gate_out, void* ws,
                            size_t ws_bytes, hipStream_t stream);

/* Bytes of workspace clearmoe_ffn_forward_padded needs for this shape (room
 * for a padded batch of E * T * k rows); 0 if the shape is invalid. */
size_t clearmoe_padded_workspace_bytes(const clearmoe_shape* shape);

/* The whole layer through the padded batched backend (Sec. III "Dispatch
 * Backends", the cuBLAS variant: expert sub-batches padded to the largest and
 * stacked into one 3-D batch; Sec. IV dispatch benchmark, Table C6).  Same
 * arguments, layouts and results as clearmoe_ffn_forward, up to rounding
 * order; it exists to measure what padding costs under imbalanced routing.
 * Route, dispatch, fc1 + GELU and the shared basis run as in the k > 1 path of
 * clearmoe_ffn_forward; then, with C the largest expert count, expert e owns
 * rows [e C, e C + C) of a padded batch, its assignments first and zero rows
 * after, and the residual products run over all E * C rows (padding rows
 * included) before the combine reads the real rows back.
 * The host needs C to size the batch: the call copies the counts to pinned
 * host memory (one small buffer per calling thread, kept until the process
 * ends) and waits for them on an event, so it blocks the calling thread until
 * dispatch has finished on the stream (fc1 and the shared basis are queued
 * first and overlap the wait), and it cannot be captured into a graph.
 * ws must hold clearmoe_padded_workspace_bytes(shape). */
int clearmoe_ffn_forward_padded(const clearmoe_shape* shape, const void* x, const void* W1,
                                const float* b1, const void* US, const void* Vt, const float* b2,
                                const void* P, const void* Q, const void* Wg, const float* bg,
                                void* y, int32_t* idx_out, float* gate_out, void* ws,
                                size_t ws_bytes, hipStream_t stream);

/* Dense comparator: y = GELU(x W1^T + b1) W2^T + b2, the unexpertised FFN the
 * paper's dense rows time (Table III, D0), run through the same GEMM kernels.
 *   x [T, D]; W1 [H, D], b1 [H]; W2 [D, H], b2 [D]; y [T, D] out (dtype).
 * Uses T, D, H, dtype (E, k, r, q must still be valid); the workspace of
 * clearmoe_workspace_bytes(shape) suffices, and so does that of a CLEAR-MoE
 * layer with the same T, D, H and dtype (only the fc1 activations are kept
 * there). */
int clearmoe_dense_ffn_forward(const clearmoe_shape* shape, const void* x, const void* W1,
                               const float* b1, const void* W2, const float* b2, void* y,
                               void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- Stage timing (measurement support) -----------------------------------
 * Kernel stages of the entry points above.  While timing is on, the kernel of
 * every timed launch of a selected stage is dispatched with two HIP events
 * (hipExtLaunchKernel) that the dispatch itself stamps at the kernel's start
 * and end, so the elapsed time is the kernel's own and no marker packet joins
 * the stream.  A timed dispatch still costs the step a few microseconds
 * (about 5 us measured on MI355X at 12608 tokens of width 384), so a benchmark times
 * a sample of the launches.  Off by default: then the entry points behave
 * exactly as documented. */
enum {
    CLEARMOE_STAGE_ROUTE = 0,          /* logits + top-k + gates + tile histogram */
    CLEARMOE_STAGE_TILE_HIST = 1,      /* tile histogram of a given idx */
    CLEARMOE_STAGE_SCAN = 2,           /* exclusive scan of tile histograms */
    CLEARMOE_STAGE_PERMUTE = 3,        /* stable permutation (+ row copy) */
    CLEARMOE_STAGE_COMBINE = 4,        /* gated inverse-permute combine */
    CLEARMOE_STAGE_FC1 = 5,            /* z = GELU(x W1^T + b1) */
    CLEARMOE_STAGE_BASIS_T = 6,        /* t = z Vt^T */
    CLEARMOE_STAGE_BASIS_H = 7,        /* h_sh = t US^T + b2 */
    CLEARMOE_STAGE_RES_U = 8,          /* u = gate * z[perm] Q_e^T (grouped) */
    CLEARMOE_STAGE_RES_H = 9,          /* h_res = u P_e^T (grouped) */
    CLEARMOE_STAGE_COMBINE_RES = 10,   /* y = h_sh + unpermuted h_res */
    CLEARMOE_STAGE_DENSE_FC2 = 11,     /* dense comparator y = z W2^T + b2 */
    CLEARMOE_STAGE_TU = 12,            /* top-1: [t|u] = z[perm] [Vt;Q_e]^T (grouped) */
    CLEARMOE_STAGE_Y = 13,             /* top-1: y[perm] = [t|u] [US|P_e]^T + b2 (grouped) */
    CLEARMOE_STAGE_FUSED_TOP1 = 14,    /* top-1 bf16: fc1+GELU, [t|u] and y in one kernel */
    CLEARMOE_STAGE_PAD_INDEX = 15,     /* padded backend: padded row maps */
    CLEARMOE_STAGE_PAIR_KEY = 16,      /* top-2: expert-pair keys and gates */
    CLEARMOE_STAGE_TU_PAIR = 17,       /* top-2: [t|u_a|u_b] grouped by expert pair */
    CLEARMOE_STAGE_Y_PAIR = 18,        /* top-2: y grouped by pair, rows scattered */
    CLEARMOE_STAGE_RESIDUAL_ADD = 19,  /* stack: x_{l+1} = x_l + f_l(x_l) */
    CLEARMOE_N_STAGES = 20
};

/* One layer of a chained FFN stack (clearmoe_stack_forward).  The paper
 * expertises the L/2 best-scoring of a ViT's L blocks (Sec. III Phase 2; six
 * of twelve for DeiT) and keeps the others dense.
 *   moe == 0: the dense FFN  f(x) = GELU(x W1^T + b1) W2^T + b2
 *             (W1 [H, D], b1 [H], W2 [D, H], b2 [D]; the other fields unused);
 *   moe == 1: a CLEAR-MoE layer with k experts per token, weights as in
 *             clearmoe_ffn_forward_ex (W1, b1, US, Vt, b2, P, Q and the router;
 *             class tokens through router.dense_stride / router.W2).
 * Every layer has the stack's T, D, H, E, r, q and dtype. */
typedef struct {
    int32_t moe;
    int32_t k;
    const void* W1;
    const float* b1;
    const void* US;
    const void* Vt;
    const float* b2;
    const void* P;
    const void* Q;
    const void* W2;
    clearmoe_router router;
} clearmoe_stack_layer;

/* Bytes of workspace clearmoe_stack_forward needs (the largest layer's
 * workspace plus three [T, D] activation buffers); 0 if the shape or a
 * layer's k is invalid or n < 1. */
size_t clearmoe_stack_workspace_bytes(const clearmoe_shape* shape,
                                      const clearmoe_stack_layer* layers, int32_t n);

/* A chain of n FFN layers, each feeding the next (multi-layer integration of
 * Sec. III Phase 2): with residual != 0 every layer adds its input back,
 * x_{l+1} = x_l + f_l(x_l) (the FFN sublayer of a transformer block with its
 * skip connection; layer norms and attention are outside this path), else
 * x_{l+1} = f_l(x_l); y = x_n.  x [T, D] in, y [T, D] out (dtype), both
 * caller-owned; x_l lives in the workspace between layers, rounded to dtype
 * like y, and f_l is rounded to dtype before the add.  All layers run on
 * `stream` in order; argument checks cover every layer before anything is
 * launched.  shape->k is ignored (each layer has its own). */
int clearmoe_stack_forward(const clearmoe_shape* shape, const clearmoe_stack_layer* layers,
                           int32_t n, int32_t residual, const void* x, void* y, void* ws,
                           size_t ws_bytes, hipStream_t stream);

/* Name of a stage (static string; "?" if out of range). */
const char* clearmoe_stage_name(int stage);

/* Start timing the stages whose bit is set in stage_mask, for at most
 * max_records launches in total (the events are created here, once).
 * Returns CLEARMOE_ERR_INVALID_ARG if timing is already on or max_records < 1,
 * CLEARMOE_ERR_HIP if an event cannot be created.  Not thread-safe. */
int clearmoe_timing_start(unsigned stage_mask, int max_records);

/* As clearmoe_timing_start, but only every every-th launch of the selected
 * stages is timed (launches 0, every, 2 every, ... counted from this call over
 * all selected stages); the others run untimed.  every >= 1, else
 * CLEARMOE_ERR_INVALID_ARG. */
int clearmoe_timing_start_sampled(unsigned stage_mask, int max_records, int every);

/* Stop timing: wait for the recorded events, then write per stage the summed
 * elapsed milliseconds (ms[CLEARMOE_N_STAGES]) and the number of timed
 * launches (launches[CLEARMOE_N_STAGES]); either pointer may be NULL.  The
 * events are destroyed and timing is off afterwards. */
int clearmoe_timing_stop(double* ms, int32_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* CLEARMOE_H */
