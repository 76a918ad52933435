/*
 * comera.h -- C ABI of the MI355X (gfx950) library for tensor-train-matrix
 * (TTM) compressed linear layers and the TTM embedding lookup of CoMERA
 * (arXiv 2405.14377).
 *
 * Formats (paper Sec. 2, eq. TTM; Sec. 3.1, eq. Wcompress):
 *   A TTM linear layer holds W in R^{N_in x N_out}, N_in = prod n_k,
 *   N_out = prod m_k, only as d cores G_k[r_{k-1}, m_k, n_k, r_k]
 *   (row-major, fp32, r_0 = r_d = 1) and d-1 rank-mask vectors D_k in R^{r_k}
 *   that sit on the bond between cores k and k+1:
 *     W[i, j] = sum_a prod_k G_k[a_{k-1}, j_k, i_k, a_k] * prod_{k<d} D_k[a_k]
 *   with i = ((i_1 n_2 + i_2) n_3 + ...) and j likewise (row-major, first
 *   factor most significant).  Factors equal to 1 are legal, so the paper's
 *   plain TT layout of Sec. 4.2 (input modes first, output modes last) is a
 *   TTM layer with unit modes.
 *
 * Operations:
 *   comera_ttm_forward   Y  = X W                    (Sec. 4.2, eq. forward)
 *   comera_ttm_backward  dX = dY W^T                 (Sec. 4.2, eq. back X)
 *                        dG_k = d<Y,dY>/dG_k          (Sec. 4.2, eq. back Gi)
 *   comera_tt_embed_forward   Y[t,:] = T[ids[t],:]    (Sec. 4.1, lookup T[I,:])
 *   comera_tt_embed_backward  dG_k = d<Y,dY>/dG_k     (linearity of the lookup)
 *   comera_ttm_plan      chooses a contraction order from the shape, ranks and
 *                        batch among the family of Prop. 4.1 (groups of
 *                        consecutive cores, then a sequential sweep of X).
 *   comera_ttm_backward_masks  the backward plus dD_k, the gradients of the
 *                        rank masks (chain rule through eq. Wcompress).
 *   comera_ttm_plan_set_fp8    the mixed-precision layer of the appendix:
 *                        the batch products on FP8 E4M3 codes, the
 *                        batch-free steps in fp32; comera_fp8_quantize is
 *                        its quantiser.
 *
 * Conventions shared by every call:
 *   - X, Y, dY, dX are row-major [b, N] in the activation dtype of the plan
 *     (fp32, or bf16 with fp32 accumulation).  Cores, masks and core
 *     gradients are always fp32.
 *   - Every device buffer (inputs, outputs, workspace) is owned by the
 *     caller.  Outputs are overwritten, never accumulated into.
 *   - Compute calls are asynchronous on `stream` (a hipStream_t passed as
 *     void*; NULL is the default stream) and never synchronise the host.
 *   - Host-detectable argument errors return a negative status before any
 *     launch; a failed launch returns COMERA_ERR_HIP.  No C++ exception
 *     crosses this boundary.
 *   - The plan is a host object owned by the library.  Only the
 *     comera_ttm_plan_set_* calls change it (host only; not concurrently
 *     with other calls on the same plan); otherwise it may be used from
 *     several streams if each stream has its own workspace.
 */
#ifndef COMERA_H
#define COMERA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    COMERA_OK = 0,
    COMERA_ERR_INVALID_ARG = -1,  /* bad shape, pointer, size or order index */
    COMERA_ERR_UNSUPPORTED = -2,  /* valid request the library cannot run (too large) */
    COMERA_ERR_WORKSPACE = -3,    /* workspace missing or smaller than required */
    COMERA_ERR_HIP = -4,          /* a HIP runtime call or kernel launch failed */
    COMERA_ERR_INTERNAL = -5
} comera_status;

typedef enum { COMERA_F32 = 0, COMERA_BF16 = 1 } comera_dtype;

#define COMERA_MAX_CORES 8

/* Order kinds reported by comera_ttm_plan_order_info (`kind`). */
#define COMERA_ORDER_DENSE 0      /* one group: rebuild W, then one GEMM per product */
#define COMERA_ORDER_SWEEP_RL 1   /* several groups, X swept from the last group */
#define COMERA_ORDER_SWEEP_LR 2   /* several groups, X swept from the first group */
#define COMERA_ORDER_ZERO 3       /* some bond has no active mask entry: W == 0 */
#define COMERA_ORDER_FUSED_RL 4   /* every core its own group, X swept from the last core by
                                     fused kernels with the per-token states in LDS */

/* Shape of one TTM linear layer (Sec. 2 eq. TTM, Sec. 4.2).
 * Core k (0-based) is G_k[r[k], m[k], n[k], r[k+1]], fp32 row-major.
 * n = input factors (N_in = prod n), m = output factors (N_out = prod m),
 * r[0] = r[d] = 1.  act = dtype of X, Y, dY, dX. */
typedef struct {
    int32_t d;
    int32_t act;                          /* comera_dtype */
    int64_t n[COMERA_MAX_CORES];
    int64_t m[COMERA_MAX_CORES];
    int64_t r[COMERA_MAX_CORES + 1];
} comera_ttm_shape;

typedef struct comera_ttm_plan_s *comera_ttm_plan_t;

/* Plan one TTM layer (Sec. 4.2, Prop. 4.1: groups of consecutive cores,
 * then a sweep of X through the groups; rank masks of eq. Wcompress).  Every
 * order of that family is enumerated and priced by a cost model (flops at
 * half the peak, HBM bytes, launches).  Host only: no device work.
 *   s            shape (validated: 1 <= d <= 8, factors >= 1, ranks >= 1,
 *                r[0] = r[d] = 1, act in {F32, BF16}).
 *   batch        number of token rows b (>= 0) the plan is sized for; calls
 *                may pass any b' <= batch.
 *   mask_active  optional host array: for bonds k = 1..d-1 in order, r[k]
 *                bytes each (concatenated); nonzero = entry may be nonzero.
 *                The caller promises D_k[a] == 0 wherever the byte is 0.
 *                NULL = every entry active.  Used to compact ranks: inactive
 *                slices are dropped from every contraction.
 *   force_order  -1 = choose the order with the least predicted time among
 *                the orders this library executes; otherwise an index in
 *                [0, comera_ttm_plan_num_orders) (COMERA_ERR_UNSUPPORTED if
 *                that order has no kernels).
 *   out          receives the plan; release it with comera_ttm_plan_destroy.
 * Orders are numbered deterministically: index 0 is the dense order (one
 * group); then for each composition of the cores into >= 2 consecutive
 * groups, in increasing order of its cut bit mask, the right-to-left sweep
 * and then the left-to-right sweep; last, the fused single-core sweep
 * (COMERA_ORDER_FUSED_RL: one forward kernel, one backward kernel plus the
 * fixed-order sum of its per-workgroup core-gradient partials; executable
 * when the per-token states fit the LDS of a CU and the compacted ranks are
 * at most 64).  d = 3 gives 8 orders, d = 4 gives 16.  Ties in predicted
 * time go to the lowest index. */
comera_status comera_ttm_plan(const comera_ttm_shape *s, int64_t batch,
                              const uint8_t *mask_active, int32_t force_order,
                              comera_ttm_plan_t *out);

/* Number of enumerated orders (2^d), or 0 for a NULL plan. */
int32_t comera_ttm_plan_num_orders(comera_ttm_plan_t p);

/* Index of the order the plan executes. */
int32_t comera_ttm_plan_chosen(comera_ttm_plan_t p);

/* Describe order i: a NUL-terminated text like "dense [0,1,2]" or
 * "sweep-rl [0][1,2]" (truncated to len bytes), its kind, its predicted
 * forward and backward flops and HBM bytes at the planned batch, and whether
 * the library has kernels for it.  Any output pointer may be NULL. */
comera_status comera_ttm_plan_order_info(comera_ttm_plan_t p, int32_t i, char *desc,
                                         size_t len, int32_t *kind, double *flops_fwd,
                                         double *flops_bwd, double *bytes,
                                         int32_t *executable);

/* Device workspace (bytes) that forward and backward need for this plan at
 * its planned batch.  Forward and backward may use the same buffer; no state
 * is carried from forward to backward unless reuse is switched on (below). */
size_t comera_ttm_workspace_bytes(comera_ttm_plan_t p);

/* Y[b, N_out] = X[b, N_in] W  (Sec. 4.2 eq. forward).
 *   X, Y   device, activation dtype, row-major, b <= planned batch.
 *   G      host array of d device pointers to the fp32 cores.
 *   D      host array of d-1 device pointers to fp32 masks, or NULL (= ones).
 *   ws     device workspace of ws_bytes >= comera_ttm_workspace_bytes. */
comera_status comera_ttm_forward(comera_ttm_plan_t p, int64_t b, const void *X,
                                 const float *const *G, const float *const *D, void *Y,
                                 void *ws, size_t ws_bytes, void *stream);

/* comera_ttm_forward for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same Y = X W with no workspace argument.  The scratch it
 * needs (folded cores, left chains, W^T) lives in one static device array of
 * COMERA_TTM_NOALLOC_SCRATCH_BYTES per GPU, reserved when the library is
 * loaded on that GPU and held until the process ends; the call allocates
 * nothing.  It runs on the current device, which must be the device of
 * `stream`.  Every call on a GPU shares that GPU's array, so calls that
 * overlap on one GPU (other streams, other threads) race: serialise them.
 * Nothing carries over between calls (every region is written before it is
 * read).  The batch product is not split over K, so results may differ
 * from comera_ttm_forward's in the last bits at small batches.
 * Errors: as comera_ttm_forward; COMERA_ERR_UNSUPPORTED for a plan whose
 * order is not the dense order (plan with force_order = 0 when the planner
 * picks a sweep), with FP8 or reuse switched on, or whose scratch (folded
 * cores + left chains + W + W^T in the activation dtype) exceeds
 * COMERA_TTM_NOALLOC_SCRATCH_BYTES. */
#define COMERA_TTM_NOALLOC_SCRATCH_BYTES (64u << 20)
comera_status comera_ttm_forward_noalloc(comera_ttm_plan_t p, int64_t b, const void *X,
                                         const float *const *G, const float *const *D, void *Y,
                                         void *stream);

/* dX[b, N_in] = dY W^T (eq. back X) and every dG_k (eq. back Gi), with
 * dG_k scaled by D_{k-1} on its left bond and D_k on its right bond (chain
 * rule through eq. Wcompress).  dX may be NULL (not computed); dG may be
 * NULL or hold NULL entries (those gradients are not computed).  dG_k is
 * written in the core's layout G_k[r_{k-1}, m_k, n_k, r_k], fp32. */
comera_status comera_ttm_backward(comera_ttm_plan_t p, int64_t b, const void *X,
                                  const void *dY, const float *const *G,
                                  const float *const *D, void *dX, float *const *dG,
                                  void *ws, size_t ws_bytes, void *stream);

/* comera_ttm_backward plus the gradients of the rank masks (chain rule
 * through eq. Wcompress, the quantity the rank-adaptive training of Sec. 3
 * updates D_k with): dD is NULL or a host array of d-1 device pointers
 * (entries may be NULL = not computed); dD_k receives r[k+1] fp32 values,
 *   dD_k[c] = <dW, dW/dD_k[c]> = sum_{a,m,n} dG~_k[a,m,n,c] G_k[a,m,n,c],
 * dG~_k being the gradient of the masked core G_k D_k.  Entries declared
 * inactive in the plan's mask_active (pruned slices, dropped from every
 * contraction) receive 0; with mask_active NULL every entry gets its exact
 * gradient, also where D_k[c] == 0.  Sums run in a fixed order (bitwise
 * repeatable).  Other arguments and errors as for comera_ttm_backward. */
comera_status comera_ttm_backward_masks(comera_ttm_plan_t p, int64_t b, const void *X,
                                        const void *dY, const float *const *G,
                                        const float *const *D, void *dX, float *const *dG,
                                        float *const *dD, void *ws, size_t ws_bytes,
                                        void *stream);

void comera_ttm_plan_destroy(comera_ttm_plan_t p);

/* Reuse of the forward's batch-free work in the backward call, as a
 * training step saves forward intermediates for its backward pass (the
 * contraction paths of Sec. 4.2 keep their forward results for the
 * gradients).  With enable != 0, comera_ttm_forward of the dense order also
 * writes W in the layout that dX reads, and comera_ttm_backward takes the
 * masked cores, left chains and W from the workspace instead of rebuilding
 * them; under a sweep order it likewise takes the group matrices and the
 * activation states of the forward sweep.  The caller then guarantees that
 * every backward call follows a forward call of this plan on the same
 * workspace with the same G, D and X, with no other call of this plan on
 * that workspace in between; otherwise the results are undefined (no error
 * can be detected).  Off by default; host only, no device work.
 * Returns COMERA_ERR_INVALID_ARG for a NULL plan. */
comera_status comera_ttm_plan_set_reuse_forward(comera_ttm_plan_t p, int32_t enable);

/* Mixed-precision layer (appendix on mixed-precision CoMERA: contractions
 * that carry the batch index run in a low precision, the batch-free ones in
 * full precision).  With enable != 0 the three batch products of the dense
 * order -- Y = X W, dX = dY W^T, dW = X^T dY -- read OCP FP8 E4M3 codes of
 * X, dY and W in the format and scaling of comera_fp8_quantize (one scale
 * per tensor and call), accumulate in fp32 and multiply by the inverse
 * scales.  W is rebuilt from the cores in fp32; the projections of dW onto
 * the cores, the mask gradients and every other batch-free step stay fp32.
 * X, Y, dY and dX keep the plan's activation dtype.  K of each product is
 * padded with zero codes to a multiple of 128.  Changes the workspace size:
 * query comera_ttm_workspace_bytes afterwards.  Combines with reuse (the
 * backward call then also takes the codes of W and X^T and their scales
 * from the forward call).  Host only, no device work.  Returns
 * COMERA_ERR_UNSUPPORTED if the plan's order is not the dense order (plan
 * with force_order = 0) or a code buffer would exceed 2^32 bytes,
 * COMERA_ERR_INVALID_ARG for a NULL plan.  Off by default. */
comera_status comera_ttm_plan_set_fp8(comera_ttm_plan_t p, int32_t enable);

/* OCP FP8 E4M3 codes of a row-major tensor x [rows, cols] (fp32 or bf16 by
 * dtype) with one power-of-two scale: s = 2^e, e the largest integer with
 * max|x| * s <= 448, clamped to [-60, 60] (s = 1 if x is all zeros); each
 * code is x * s (exact in fp32) rounded to the nearest E4M3 value, ties to
 * the even code, magnitudes above 448 saturated to 448, the sign bit kept
 * (also where the value rounds to zero).  Inputs must be finite.
 *   q      device [rows, ldq] codes of x, or NULL; columns cols..ldq-1 get 0.
 *   qt     device [cols, ldt] codes of x^T, or NULL; columns rows..ldt-1 get 0.
 *   scale  device float[1], receives s (x ~ value(code) / s).
 *   ws     device scratch of ws_bytes >= COMERA_FP8_QUANTIZE_WS_BYTES.
 * At least one of q, qt; ldq >= cols, ldt >= rows.  rows or cols == 0:
 * nothing is written.  Asynchronous on stream. */
#define COMERA_FP8_QUANTIZE_WS_BYTES 2048
comera_status comera_fp8_quantize(const void *x, int32_t dtype, int64_t rows, int64_t cols,
                                  uint8_t *q, int64_t ldq, uint8_t *qt, int64_t ldt,
                                  float *scale, void *ws, size_t ws_bytes, void *stream);

/* Early-stage regulariser gradients (Sec. 3.2, eq. pretrain-rank), added in
 * place, on `stream`, to the loss gradients a backward call returned:
 *   dG_k += 2 beta G_k                         (beta ||G||^2, every core)
 *   dD_k[c] += gamma sign(D_k[c]) (l_k + r_k)  (gamma S^(D), every bond)
 * S^ is the layer size with each ||D_k||_0 relaxed to ||D_k||_1, s_j = m_j n_j;
 * l_k = s_k for k = 0, else s_k ||D_{k-1}||_1; r_k = s_{k+1} for k + 1 = d - 1,
 * else s_{k+1} ||D_{k+1}||_1; sign(0) = 0.  G, dG: d device pointers to fp32
 * cores [r[k], m[k], n[k], r[k+1]] (dG null, or an entry null: that core is
 * skipped); D, dD: d - 1 device pointers to fp32 masks of length r[k+1] (dD
 * null or an entry null: skipped; any dD needs every D).  Caller owns all
 * memory; nothing is allocated.  Errors: bad shape, negative or non-finite
 * gamma / beta, a dG without its G, a dD without every D -> INVALID_ARG; a
 * core above 2^31 entries -> UNSUPPORTED; launch failure -> HIP.
 * Deterministic: the l1 norms are summed in a fixed order. */
comera_status comera_ttm_regularizer_grads(const comera_ttm_shape *s, float gamma, float beta,
                                           const float *const *G, const float *const *D, float *const *dG,
                                           float *const *dD, void *stream);

/* Diagnostics: per-kernel timing of the batch products of a plan.  While
 * enabled, forward and backward record a pair of HIP events on the call's
 * stream around each launch of the kernels below; comera_ttm_plan_kernel_time
 * waits for the recorded events (a host synchronisation), returns the mean
 * duration in ms and the number of launches since the last query, and
 * clears the record.  Meant for one stream at a time; off by default. */
#define COMERA_KERNEL_FWD 0   /* Y = X W */
#define COMERA_KERNEL_DX 1    /* dX = dY W^T */
#define COMERA_KERNEL_DW 2    /* dW = X^T dY (all splits) */
comera_status comera_ttm_plan_set_timing(comera_ttm_plan_t p, int32_t enable);
comera_status comera_ttm_plan_kernel_time(comera_ttm_plan_t p, int32_t kernel, double *avg_ms,
                                          int32_t *count);

/* Shape of a TTM embedding table T[V, E] (Sec. 4.1): V = prod v (rows,
 * vocabulary), E = prod e (embedding width).  Core k is
 * G_k[r[k], v[k], e[k], r[k+1]] (row factor second), fp32, r[0] = r[d] = 1.
 * A row id is split into digits z_k row-major (first factor most
 * significant): id = ((z_1 v_2 + z_2) v_3 + z_3) ... */
typedef struct {
    int32_t d;
    int32_t pad_;
    int64_t v[COMERA_MAX_CORES];
    int64_t e[COMERA_MAX_CORES];
    int64_t r[COMERA_MAX_CORES + 1];
} comera_tt_embed_shape;

/* Workspace bytes for n_tokens ids (forward and backward; the same size
 * serves both). */
size_t comera_tt_embed_workspace_bytes(const comera_tt_embed_shape *s, int64_t n_tokens);

/* Y[t, :] = T[ids[t], :] for t < n_tokens (Sec. 4.1, eq. emb_A1/emb_A2/
 * emb_unique: a prefix table over the leading digits, then one small
 * contraction per row).
 *   ids       device int64 [n_tokens]; contract 0 <= id < V.
 *   G, D      as for the linear layer (D may be NULL).
 *   Y         device fp32 [n_tokens, E].
 *   err_flag  device int32 or NULL: set to 1 if some id is out of range
 *             (those rows are written as zeros); never cleared by the call. */
comera_status comera_tt_embed_forward(const comera_tt_embed_shape *s, const int64_t *ids,
                                      int64_t n_tokens, const float *const *G,
                                      const float *const *D, float *Y, void *ws,
                                      size_t ws_bytes, int32_t *err_flag, void *stream);

/* dG_k = d<Y, dY>/dG_k for every core (scaled by the masks as in the
 * linear layer), from dY device fp32 [n_tokens, E].  Tokens are grouped by
 * id with a stable sort and every sum runs in a fixed order, so the result
 * is bitwise reproducible for any `deterministic` value (the flag is
 * accepted for interface stability).  Out-of-range ids contribute nothing
 * and set *err_flag.  dG entries must all be non-NULL. */
comera_status comera_tt_embed_backward(const comera_tt_embed_shape *s, const int64_t *ids,
                                       int64_t n_tokens, const float *dY,
                                       const float *const *G, const float *const *D,
                                       float *const *dG, int32_t deterministic, void *ws,
                                       size_t ws_bytes, int32_t *err_flag, void *stream);

/* comera_tt_embed_backward with options.  flags: bitwise OR of
 *   COMERA_EMBED_REUSE_FORWARD  take the masked prefix cores and the prefix
 *       table from the workspace, where the last comera_tt_embed_forward
 *       call with this workspace, the same shape, n_tokens, G and D left
 *       them (a training step's forward then backward); otherwise the
 *       results are undefined (no error can be detected).
 * Unknown flag bits are an error (COMERA_ERR_INVALID_ARG). */
#define COMERA_EMBED_REUSE_FORWARD 1
comera_status comera_tt_embed_backward_ex(const comera_tt_embed_shape *s, const int64_t *ids,
                                          int64_t n_tokens, const float *dY,
                                          const float *const *G, const float *const *D,
                                          float *const *dG, int32_t flags, void *ws,
                                          size_t ws_bytes, int32_t *err_flag, void *stream);

/* Diagnostics for host-side tests, usable without a GPU: launch check
 * mode.  While enabled, every compute call of this library runs its whole
 * host path (argument checks, plan and workspace arithmetic, launch sizing)
 * but, instead of launching each kernel, checks its configuration against
 * the gfx950 limits (grid x in [1, 2^31 - 1], grid y and z in [1, 65535],
 * 1 to 1024 threads per workgroup, at most 160 KiB of LDS) and records it.
 * No device memory is read or written, so outputs are left as they were; a
 * configuration outside the limits makes the call return COMERA_ERR_HIP.
 * The mode is process-wide: do not make real compute calls from other
 * threads while it is on.  Each call of comera_debug_launch_check clears the
 * record.  comera_debug_launch_info describes record i (name = the kernel
 * expression as written in the source); any output pointer may be NULL. */
comera_status comera_debug_launch_check(int32_t enable);
int32_t comera_debug_launch_count(void);
comera_status comera_debug_launch_info(int32_t i, char *name, size_t len, uint32_t *grid3, uint32_t *block3,
                                       uint64_t *lds, int32_t *ok);

/* Static English text for a status code. */
const char *comera_status_string(comera_status s);

/* The HIP error behind the last COMERA_ERR_HIP returned on the calling
 * thread: its HIP name and the step that reported it ("" if none).  The
 * text stays valid until the next failing call on the same thread. */
const char *comera_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* COMERA_H */
