/*
 * moce.h -- C ABI of the MI355X (gfx950) Mixture of Channel Experts forward
 * pass (arxiv 2608.23794, "Mixture of Channel Experts: Static Sparse Supports
 * with Input-Adaptive Mixing for Pointwise Projections").
 *
 * A MoCE layer replaces a pointwise projection from C input channels to E <= C
 * outputs (Sec. 3.1): E-1 routed experts, each a convex mixture of k input
 * channels on a static support (Sec. 3.2-3.3), plus one residual output that
 * averages the channels outside every support (Sec. 3.4, Eq. 6).
 *
 * Conventions shared by every entry point
 *  - The descriptor and gate structs are host memory; every array argument is
 *    a device pointer (hipMalloc'd or otherwise device-accessible) unless its
 *    name ends in _host.  The caller owns all memory.  The library never
 *    allocates device memory and keeps no pointer after a call returns.
 *  - Every call except moce_support_prepare is asynchronous on `stream`
 *    (0 = the null stream) and returns as soon as its kernels are enqueued.
 *  - Layouts: MOCE_NCHW is x[B][C][H][W] and y[B][E][H][W]; MOCE_NHWC is
 *    x[B][H][W][C] and y[B][H][W][E].  Token inputs x[B][N][C] are MOCE_NHWC
 *    with H = N, W = 1.  y always has the layout and element type of x.
 *  - Element types: x and y are both MOCE_F32 or both MOCE_BF16 (bfloat16 bit
 *    patterns, 2 bytes).  Accumulation is float32 throughout; bf16 outputs are
 *    rounded to nearest, ties to even.  d, tau, alpha and all parameters are
 *    float32; supports are int32 channel indices.
 *  - Output channel E-1 is the residual expert; channels 0..E-2 are the routed
 *    experts in support-row order.
 *  - x and y must be 16-byte aligned.
 *  - Errors are negative moce_status codes.  Every error detectable on the host
 *    is reported before anything is enqueued, and then no output is written.
 *    A failed kernel launch returns MOCE_ERR_DEVICE.  The library holds no
 *    mutable global state; calls on different streams are independent as long
 *    as their output buffers do not overlap.
 */
#ifndef MOCE_H
#define MOCE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum moce_status {
    MOCE_OK = 0,
    MOCE_ERR_NULL = -1,        /* a required pointer is NULL */
    MOCE_ERR_SHAPE = -2,       /* B, C, H, W < 1; E outside [1, C]; k outside [1, C] */
    MOCE_ERR_DTYPE = -3,       /* unknown element type or x/y types differ */
    MOCE_ERR_LAYOUT = -4,      /* unknown layout code */
    MOCE_ERR_SUPPORT = -5,     /* a support row is invalid (moce_support_prepare) */
    MOCE_ERR_GATE = -6,        /* unknown gate kind, or tau_min/tau_max invalid */
    MOCE_ERR_WORKSPACE = -7,   /* workspace NULL or smaller than required */
    MOCE_ERR_ALIGN = -8,       /* x or y not 16-byte aligned */
    MOCE_ERR_DEVICE = -9,      /* a HIP call or kernel launch failed */
    MOCE_ERR_UNSUPPORTED = -10 /* the shape exceeds a documented size limit */
} moce_status;

enum { MOCE_F32 = 0, MOCE_BF16 = 1 };
enum { MOCE_NCHW = 0, MOCE_NHWC = 1 };

/* Gate kinds.  Both read the k descriptors of an expert's support in
 * canonical order (descending routing logit), so gate position i is the
 * expert's i-th most preferred channel (Sec. 3.3).
 *  MOCE_GATE_SOFTPLUS_LINEAR: tau[b][o] = softplus(c[o] + sum_i a[o][i] d[b][s[o][i]]) + 1e-3,
 *     a per-expert linear gate (a: [E-1][k], c: [E-1]).
 *  MOCE_GATE_MLP_SIGMOID: the paper's gate (Sec. 3.3 Eq. 3): one two-layer MLP
 *     of hidden width k shared by all experts of the layer,
 *     h = ReLU(W1 z + b1), g = w2 . h + b2,
 *     tau = tau_min + (tau_max - tau_min) sigmoid(g)
 *     (W1: [k][k] row-major, row j feeds hidden unit j; b1, w2: [k]). */
enum { MOCE_GATE_SOFTPLUS_LINEAR = 0, MOCE_GATE_MLP_SIGMOID = 1 };

typedef struct moce_desc {
    int64_t B, C, H, W;   /* x is B images of C channels over H*W positions */
    int32_t E;            /* outputs: E-1 routed experts + 1 residual, 1 <= E <= C */
    int32_t k;            /* support size, 1 <= k <= C */
    int32_t x_dtype;      /* MOCE_F32 or MOCE_BF16 */
    int32_t y_dtype;      /* must equal x_dtype */
    int32_t layout;       /* MOCE_NCHW or MOCE_NHWC */
    int32_t reserved;     /* set to 0 */
} moce_desc;

typedef struct moce_gate_params {
    int32_t kind;         /* MOCE_GATE_* */
    int32_t reserved;     /* set to 0 */
    const float* a;       /* softplus-linear: [E-1][k] slopes, canonical positions */
    const float* c;       /* softplus-linear: [E-1] offsets */
    const float* W1;      /* MLP: [k][k] */
    const float* b1;      /* MLP: [k] */
    const float* w2;      /* MLP: [k] */
    float b2;             /* MLP: output bias */
    float tau_min;        /* MLP: lower temperature bound, > 0 */
    float tau_max;        /* MLP: upper temperature bound, >= tau_min */
} moce_gate_params;

/* Static support preparation (Sec. 3.2 Eq. 2: supports fixed at inference;
 * Sec. 3.3: gate input order; Sec. 3.4: the uncovered set U).
 *
 * In:  s[E-1][k] int32 channel indices and w[E-1][k] float32 selected routing
 *      logits, one row per routed expert, in any order.
 * Out: s_out, w_out [E-1][k]: each row sorted by logit descending, equal
 *      logits by ascending channel (the canonical order every other entry
 *      point expects); covered[C] uint8: 1 if the channel is in some support;
 *      U[C] int32: the uncovered channels ascending in U[0..nU-1] (the rest
 *      is left unspecified); info[2] int32 device scratch receiving
 *      {nU, first bad expert or -1}; *nU_host and *bad_expert_host receive the
 *      same two values.
 * A row is invalid if a channel lies outside [0, C), repeats within the row,
 * or its logit is not finite; the call then returns MOCE_ERR_SUPPORT with
 * *bad_expert_host = the lowest invalid expert (outputs other than info and
 * the two host values are unspecified).  s_out/w_out may not alias s/w.
 * This call synchronises `stream` once (it is a once-per-model step).
 * Limits: C <= 2^24, k <= 4096. */
moce_status moce_support_prepare(const moce_desc* desc, const int32_t* s, const float* w,
                                 int32_t* s_out, float* w_out, uint8_t* covered, int32_t* U,
                                 int32_t* info, int32_t* nU_host, int32_t* bad_expert_host,
                                 hipStream_t stream);

/* moce_support_prepare for supports kept in the deployment storage format:
 * s[E-1][k] as 16-bit unsigned channel indices (Sec. 3.5, Storage: a
 * deployed layer keeps its (E-1)k selected logits, their indices in 16 bits
 * and the gate).  Same outputs (int32 prepared rows), checks and errors;
 * MOCE_ERR_UNSUPPORTED when C > 65536.  This call synchronises `stream`
 * once. */
moce_status moce_support_prepare16(const moce_desc* desc, const uint16_t* s, const float* w,
                                   int32_t* s_out, float* w_out, uint8_t* covered, int32_t* U,
                                   int32_t* info, int32_t* nU_host, int32_t* bad_expert_host,
                                   hipStream_t stream);

/* Global average pooling descriptor z = GAP(x) (Sec. 3.3):
 * d[b][c] = (1 / (H W)) sum over positions of x[b][c][.]; d is [B][C] float32. */
moce_status moce_pool(const moce_desc* desc, const void* x, float* d, hipStream_t stream);

/* Temperatures (Sec. 3.3, Eq. 3 or the softplus-linear form) and mixing
 * coefficients (Eq. 4): tau[b][o] and, if alpha != NULL,
 * alpha[b][o][i] = exp(w[o][i] / tau[b][o]) / sum_j exp(w[o][j] / tau[b][o]).
 * d is [B][C]; s, w are prepared rows; tau is [B][E-1]; alpha is [B][E-1][k].
 * Does nothing when E == 1.  Limits for MOCE_GATE_MLP_SIGMOID: k <= 256. */
moce_status moce_gate(const moce_desc* desc, const float* d, const int32_t* s, const float* w,
                      const moce_gate_params* gate, float* tau, float* alpha, hipStream_t stream);

/* Temperatures, coefficients and mixing in one kernel (Secs. 3.3-3.4): the
 * y of moce_gate followed by moce_mix, bit for bit, from the pooled
 * descriptors d [B][C], without writing tau or alpha.  Each workgroup of the
 * mix evaluates the softplus-linear gate for the experts of the images it
 * mixes.  Only where moce_forward_path(desc, gate->kind) is
 * MOCE_PATH_MFMA_GATE (otherwise MOCE_ERR_UNSUPPORTED); s, w: prepared rows;
 * U, nU as for moce_mix; y is fully overwritten. */
moce_status moce_gate_mix(const moce_desc* desc, const void* x, const float* d, const int32_t* s, const float* w,
                          const moce_gate_params* gate, const int32_t* U, int32_t nU, void* y,
                          hipStream_t stream);

/* Routed outputs (Sec. 3.3 Eq. 5) and residual output (Sec. 3.4 Eq. 6):
 * y[b][o][p] = sum_i alpha[b][o][i] x[b][s[o][i]][p] for o < E-1, and
 * y[b][E-1][p] = (1/nU) sum_{c in U} x[b][c][p], or 0 when nU == 0.
 * s: prepared [E-1][k]; alpha: [B][E-1][k]; U: [nU] uncovered channels with
 * 0 <= nU <= C (U may be NULL when nU == 0).  y is fully overwritten. */
moce_status moce_mix(const moce_desc* desc, const void* x, const int32_t* s, const float* alpha,
                     const int32_t* U, int32_t nU, void* y, hipStream_t stream);

/* Bytes of device workspace moce_forward needs for `desc` (0 on an invalid
 * descriptor).  The workspace holds the descriptor d, the temperatures, the
 * softmax statistics and, depending on the path, the coefficients or the
 * support schedule. */
size_t moce_forward_workspace_bytes(const moce_desc* desc);

/* Paths moce_forward can take. */
enum { MOCE_PATH_GENERIC = 0, MOCE_PATH_TILE = 1, MOCE_PATH_MFMA = 2, MOCE_PATH_MFMA_GATE = 3,
       MOCE_PATH_SCHEDULED = 4, MOCE_PATH_GATHER = 5 };

/* The path moce_forward takes for `desc` (moce_mix takes the same kernels,
 * MOCE_PATH_MFMA for MOCE_PATH_MFMA_GATE, MOCE_PATH_GENERIC for
 * MOCE_PATH_SCHEDULED, the gather for MOCE_PATH_GATHER):
 *  MOCE_PATH_GATHER: channels-last bfloat16 with small supports (k <= 16,
 *     C a multiple of 8 up to 4096, E-1 <= 1024, or 512 for k > 8): pooling, the gate's
 *     coefficients, then a gather whose work scales with k (x staged in LDS
 *     transposed, 8 positions per read);
 *  MOCE_PATH_SCHEDULED: channels-last bfloat16 (C a multiple of 64 up to
 *     4096, E a multiple of 8): pooling, the gate's softmax statistics, then
 *     a schedule of the supports by 64-channel step (Sec. 3.2: static
 *     supports) and the routed and residual outputs as a dense bf16 product
 *     on the matrix cores whose coefficient operand is written step by step
 *     from the schedule (coefficients split into two bf16 parts: 16
 *     significant bits);
 *  MOCE_PATH_MFMA_GATE: MOCE_PATH_MFMA with the softplus-linear gate
 *     evaluated inside the mix kernel, as moce_gate_mix (k = 32);
 *  MOCE_PATH_MFMA: the gate kernel, then the routed and residual outputs of an image as one dense
 *     bf16 matrix product on the matrix cores, the coefficients split into
 *     bf16 parts that sum to them exactly (NCHW bfloat16, E-1 >= 1, C a
 *     multiple of 32 up to 256, E <= 64, H*W a multiple of 8);
 *  MOCE_PATH_TILE: the tile gather kernel (NCHW bfloat16, C <= 256, H*W a
 *     multiple of 8);
 *  MOCE_PATH_GENERIC: the layout- and type-generic kernels.
 * All compute the same values up to float32 rounding order; the MFMA path
 * requires distinct channels within each support row, as
 * moce_support_prepare guarantees.  `gate_kind` must be a valid gate kind.
 * A negative moce_status for an invalid descriptor or gate kind. */
int moce_forward_path(const moce_desc* desc, int gate_kind);

/* The whole layer (Secs. 3.3-3.4): pooling, temperatures, mixing
 * coefficients, routed experts and residual, equal to moce_pool + moce_gate +
 * moce_mix.  s, w: prepared rows; U, nU: as returned by moce_support_prepare;
 * ws: device workspace of at least moce_forward_workspace_bytes(desc) bytes,
 * 256-byte aligned, owned by the caller; its contents on entry are ignored and
 * on return unspecified.  Concurrent calls must use distinct workspaces. */
moce_status moce_forward(const moce_desc* desc, const void* x, const int32_t* s, const float* w,
                         const moce_gate_params* gate, const int32_t* U, int32_t nU, void* y,
                         void* ws, size_t ws_bytes, hipStream_t stream);

/* Output epilogue of moce_forward_ex: each output value v of channel o
 * (routed or residual) becomes act(scale[o] v + shift[o]) before it is
 * rounded and stored, act = ReLU when relu != 0 and the identity otherwise.
 * scale, shift: device float32 [E], both given or both NULL (no affine map).
 * The replaced projection is followed by batch normalisation and the block's
 * nonlinearity, which the paper leaves unchanged (Sec. 4.1); at inference the
 * normalisation is this affine map (scale = gamma / sqrt(var + eps),
 * shift = beta - mean scale), and applying it as the output is written avoids
 * a second pass over y, the memory-traffic fusion Sec. 4.7 points to. */
typedef struct moce_epilogue {
    const float* scale;
    const float* shift;
    int32_t relu;
    int32_t reserved;     /* set to 0 */
} moce_epilogue;

/* moce_forward followed by the epilogue `ep` (NULL: none, then identical to
 * moce_forward).  On the matrix-core paths (MOCE_PATH_MFMA, MOCE_PATH_MFMA_GATE,
 * MOCE_PATH_SCHEDULED) and MOCE_PATH_GATHER the mix kernel applies it to the float32 accumulators
 * before rounding; on the others a second kernel applies it to y in place
 * (for bf16 y, to the rounded value).  Errors: those of moce_forward, and
 * MOCE_ERR_NULL when exactly one of scale and shift is NULL. */
moce_status moce_forward_ex(const moce_desc* desc, const void* x, const int32_t* s, const float* w,
                            const moce_gate_params* gate, const int32_t* U, int32_t nU, const moce_epilogue* ep,
                            void* y, void* ws, size_t ws_bytes, hipStream_t stream);

/* Bytes of the device array that moce_forward_static uses as its workspace. */
#define MOCE_STATIC_SCRATCH_BYTES ((size_t)16 << 20)

/* The whole layer, as moce_forward, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): no workspace argument and no allocation.  The
 * workspace is a fixed array of MOCE_STATIC_SCRATCH_BYTES inside the library,
 * one per GPU, held from the library's load until the process ends; its
 * device address is looked up on the first call on each device.  Same
 * arguments, kernels and results as moce_forward.  Errors: those of
 * moce_forward, and MOCE_ERR_WORKSPACE (before any launch) when
 * moce_forward_workspace_bytes(desc) exceeds MOCE_STATIC_SCRATCH_BYTES;
 * MOCE_ERR_DEVICE if the array's address cannot be obtained.  Every call on
 * one GPU shares that array: calls that overlap on the same device (on
 * different streams or from different host threads) race, and the caller
 * must serialise them. */
moce_status moce_forward_static(const moce_desc* desc, const void* x, const int32_t* s, const float* w,
                                const moce_gate_params* gate, const int32_t* U, int32_t nU, void* y,
                                hipStream_t stream);

/* Router of the input-conditioned support variant (Sec. 4.5 Eq. 11).  From the
 * pooled descriptor z of an example, h = ReLU(Wh z + bh) (d values), and the
 * example's routing logits are L(X)[e][c] = L[e][c] + sum_t q[e][t] h[t] v[c][t]
 * over the full static routing logits L[E-1][C]. */
typedef struct moce_router {
    int32_t d;            /* bottleneck width, 1 <= d <= 64 */
    int32_t reserved;     /* set to 0 */
    const float* Wh;      /* [d][C] */
    const float* bh;      /* [d] */
    const float* v;       /* [C][d] channel embeddings */
    const float* q;       /* [E-1][d] expert embeddings */
} moce_router;

/* Bytes of device workspace moce_forward_dynamic needs (0 on an invalid
 * descriptor or router width). */
size_t moce_forward_dynamic_workspace_bytes(const moce_desc* desc, int32_t d);

/* The layer with input-conditioned supports (Sec. 4.5 Eq. 11), inference path.
 * Per example b: z = GAP(x_b); L(X) as above; S_e(X) = the k channels of
 * largest L(X)[e][.], equal logits by ascending channel, in canonical order
 * (logit descending, then channel ascending); the gate reads z at S_e(X) in
 * that order (gate position i is the i-th channel of S_e(X)); the
 * coefficients are the softmax of L(X)[e][S_e(X)] over the temperature; the
 * residual output E-1 is the mean of x over U(X), the channels in no
 * S_e(X) of that example (0 when U(X) is empty).
 *
 * x, y as for moce_forward (16-byte aligned, y fully overwritten);
 * L: [E-1][C] float32 device; router: host struct of device pointers;
 * gate: as for moce_forward (gate->a indexed by canonical position);
 * S_out: optional device [B][E-1][k] int32 receiving S_e(X) (NULL: not
 * written); ws: device workspace of at least
 * moce_forward_dynamic_workspace_bytes(desc, router->d) bytes, 256-byte
 * aligned, contents on return unspecified.
 * Errors: those of moce_forward; MOCE_ERR_NULL for a missing L, router or
 * router array; MOCE_ERR_UNSUPPORTED when d > 64, k > 512 or C > 4096.
 * Asynchronous on `stream`. */
moce_status moce_forward_dynamic(const moce_desc* desc, const void* x, const float* L, const moce_router* router,
                                 const moce_gate_params* gate, void* y, int32_t* S_out, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/* Gradient outputs of the gate's parameters (device arrays, float32, fully
 * overwritten); only those of the gate's own kind are read and written.
 *  MOCE_GATE_SOFTPLUS_LINEAR: da [E-1][k] (canonical positions, as a), dc [E-1];
 *  MOCE_GATE_MLP_SIGMOID: dW1 [k][k], db1 [k], dw2 [k], db2 [1]. */
typedef struct moce_gate_grads {
    float* da;
    float* dc;
    float* dW1;
    float* db1;
    float* dw2;
    float* db2;
} moce_gate_grads;

/* Bytes of device workspace moce_backward needs for `desc` with a gate of
 * kind `gate_kind` (0 on an invalid descriptor or kind, or a shape beyond the
 * backward's limits). */
size_t moce_backward_workspace_bytes(const moce_desc* desc, int gate_kind);

/* Gradients of the static layer (Secs. 3.2-3.4) for an upstream gradient dy
 * of y = moce_forward(x).  The supports are fixed (Sec. 3.2: no gradient
 * through the selection); the loss reaches the routing logits only through
 * the selected values w (Eq. 4), the gate through the temperature, and x
 * both through the routed and residual sums (Eqs. 5-6) and through the
 * pooled descriptor that feeds the gate (Sec. 3.3):
 *   dx:  d loss / d x, layout and element type of x, fully overwritten;
 *   dw:  [E-1][k] float32, d loss / d w[e][i] for the prepared rows
 *        (canonical order), fully overwritten;
 *   the gate's parameter gradients into *grads (moce_gate_grads).
 * x, s, w, gate as for moce_forward (prepared rows; the uncovered set is
 * derived from s); dy: the layout and element type of y; x, dy and dx
 * 16-byte aligned; ws: device workspace of at least
 * moce_backward_workspace_bytes(desc, gate->kind) bytes, 256-byte aligned,
 * contents on return unspecified.  Gradients are accumulated in float32.
 * Errors: those of moce_forward; MOCE_ERR_NULL for a missing dy, dx, dw or
 * gradient array of the gate's kind; MOCE_ERR_UNSUPPORTED when k > 1024, or
 * k > 128 with the MLP gate.  Asynchronous on `stream`. */
moce_status moce_backward(const moce_desc* desc, const void* x, const void* dy, const int32_t* s, const float* w,
                          const moce_gate_params* gate, void* dx, float* dw, const moce_gate_grads* grads,
                          void* ws, size_t ws_bytes, hipStream_t stream);

/* Bytes of device workspace moce_logit_backward needs (0 when R < 1 or C is
 * outside [1, 32768]). */
size_t moce_logit_backward_workspace_bytes(int32_t R, int64_t C);

/* The coverage loss over the full routing logits (Sec. 3.4 Eq. 7) and the
 * whole gradient of the routing logits (Sec. 3.2: the task loss reaches the
 * selected entries, the coverage term every entry):
 *   p[e][c] = softmax_c(L[e]), u[c] = (1/R) sum_e p[e][c], ub = mean_c u[c],
 *   loss = sum_c (u[c] - ub)^2 / (ub^2 + eps),
 *   dL[e][c] = lambda d loss / d L[e][c] + (dw[e][i] where c = s[e][i]).
 * L: [R][C] float32 (R = E-1 routed experts); s, dw: prepared rows and the
 * dw of moce_backward, [R][k], or both NULL for the coverage term alone;
 * loss: device float, or NULL; dL: [R][C] float32, fully overwritten;
 * eps >= 0 (the paper leaves it unstated); ws as sized above.
 * Errors: MOCE_ERR_NULL (L, dL, ws; s without dw or dw without s),
 * MOCE_ERR_SHAPE (R < 1, C < 1, k outside [1, C] with dw given),
 * MOCE_ERR_UNSUPPORTED (C > 32768), MOCE_ERR_WORKSPACE, MOCE_ERR_ALIGN
 * (ws not 256-byte aligned); eps < 0 or not finite: MOCE_ERR_SHAPE. */
moce_status moce_logit_backward(int32_t R, int64_t C, int32_t k, const float* L, const int32_t* s, const float* dw,
                                float eps, float lambda, float* loss, float* dL, void* ws, size_t ws_bytes,
                                hipStream_t stream);

/* Static string naming a status code. */
const char* moce_status_str(int status);

/* ABI version of this header: 1. */
int moce_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MOCE_H */
