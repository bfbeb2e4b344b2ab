/*
 * lirpa.h -- C ABI of the MI355X (gfx950) batched LiRPA bound library.
 *
 * Computes sound lower bounds of linear properties of a ReLU network over an l_inf input box,
 * for a whole batch of branch-and-bound sub-domains at once: backward-mode linear relaxation
 * based perturbation analysis (CROWN) as described in Xu et al., "Fast and Complete: Enabling
 * Complete Neural Network Verification with Rapid and Massively Parallel Incomplete Verifiers"
 * (ICLR 2021), Sec. 2.3 (Eq. 2-7) and Sec. 3.1 (Eq. 8-9, ReLU split constraints).
 *
 * Conventions shared by every call
 * --------------------------------
 * - All tensor arguments are DEVICE pointers owned by the caller; the library reads them
 *   during the enqueued work only and never keeps them past the call (except the weights
 *   borrowed by a lirpa_net, which must outlive it).  The library never allocates or frees
 *   device memory: every scratch buffer comes from the caller's workspace `ws`.
 * - Calls validate their arguments on the host, enqueue kernels on `stream` and return without
 *   synchronising.  Return 0 (LIRPA_OK) on success, a negative lirpa_status otherwise, and
 *   lirpa_last_error() returns a thread-local message.  On EINVAL, ENOMEM, EUNSUPPORTED and
 *   EDATA nothing is enqueued.  On EDEVICE (a launch or runtime call failed part-way) the work
 *   of the call up to the failure may already be enqueued: the outputs, and the in/out
 *   optimiser state (alpha, adam_m, adam_v) of lirpa_optimize, are then undefined.
 * - Flattening is C order: a conv activation is [C][H][W]; a Linear layer after a conv reads the
 *   flattened [C][H][W] vector.  Per-neuron arrays (split, alpha, l, u, gradients) concatenate
 *   the ReLU layers 1..L-1 in layer order: n_relu = sum_{m<L} n_m values per sub-domain.
 * - Floating point is fp32 (round to nearest).  Device contents are not validated by default: a
 *   split value outside {-1, 0, 1} or an alpha outside [0, 1] gives undefined (but
 *   memory-safe) results.  With the environment variable LIRPA_VALIDATE=1 every call also
 *   enqueues a read-only check of its device inputs (split in {-1, 0, 1} as the split
 *   constraints of Sec. 3.1 require, alpha in [0, 1] as Eq. 5 requires, x0 and C finite);
 *   the findings are reported by the NEXT call on the same device, which then synchronises
 *   its stream, returns LIRPA_EDATA without enqueuing anything, names the offending input in
 *   lirpa_last_error() and clears the findings.
 */
#ifndef LIRPA_H_
#define LIRPA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LIRPA_OK = 0,
  LIRPA_EINVAL = -1,      /* bad argument: shape, null pointer, eps, S, B            */
  LIRPA_ENOMEM = -2,      /* the workspace cannot hold even one sub-domain            */
  LIRPA_EDEVICE = -3,     /* a HIP launch or runtime call failed                      */
  LIRPA_EUNSUPPORTED = -4, /* a layer shape outside the supported set                 */
  LIRPA_EDATA = -5         /* LIRPA_VALIDATE=1: the previous call's device inputs were
                              out of range (see the conventions above)                 */
} lirpa_status;

typedef enum { LIRPA_LINEAR = 0, LIRPA_CONV2D = 1 } lirpa_layer_kind;

/* One affine layer T_m: h^(m) = W g^(m-1) + b (Sec. 2.1; the paper drops biases for brevity,
 * they are kept here).  ReLU follows every layer except the last.
 * LINEAR : in_c = input features, out_c = output features, in_h = in_w = out_h = out_w = 1;
 *          W is [out_c][in_c] row-major.
 * CONV2D : cross-correlation with zero padding, W is [out_c][in_c][k][k], b is per output
 *          channel, out_h = (in_h + 2 pad - k) / stride + 1 (same for w).
 * W and b are device pointers borrowed by the net. */
typedef struct {
  int kind;
  int in_c, in_h, in_w;
  int out_c, out_h, out_w;
  int k, stride, pad;
  const float* W;
  const float* b;
} lirpa_layer;

typedef struct lirpa_net lirpa_net; /* opaque host object */

/* The network f of Sec. 2.1: affine layers T_1..T_L with a ReLU after each but the last.
 * Build it from n_layers >= 1 layers (copied; W/b pointers borrowed).  EINVAL if the
 * chain is inconsistent (n_in of T_m != n_out of T_{m-1}, a conv output size that does not
 * follow the formula above, null W/b) and EUNSUPPORTED for shapes the kernels do not handle
 * (kernel size > 7, stride > 4, more than 32 layers). */
int lirpa_net_create(const lirpa_layer* layers, int n_layers, lirpa_net** out);
void lirpa_net_destroy(lirpa_net* net);

/* n_relu = sum over the ReLU layers 1..L-1 of Sec. 2.1 of their sizes; -1 for a null net. */
int64_t lirpa_net_num_relu(const lirpa_net* net);

/* Workspace bytes for one call processing up to B_chunk sub-domains at a time with S spec
 * rows (the batch of sub-domains of Sec. 3.3 is bounded by memory).  mode 0 = lirpa_bound,
 * 1 = lirpa_bound_grad / lirpa_optimize, 2 = lirpa_bound_ul, 3 = lirpa_optimize_ul (other
 * values: 0).  A call given a smaller workspace processes its
 * batch in chunks of as many sub-domains as fit.  Returns 0 for invalid arguments and
 * SIZE_MAX when a chunk of B_chunk sub-domains cannot run at all (one bound-matrix slab would
 * exceed 2^31 floats, the kernels' 32-bit element offsets); a call then uses smaller chunks. */
size_t lirpa_workspace_bytes(const lirpa_net* net, int S, int B_chunk, int mode);

/* Batched bound (Sec. 2.3 Eq. 2-7, concretised by Eq. 8; split constraints of Sec. 3.1).
 *   x0      [n0]          centre of the box ||x - x0||_inf <= eps (eps >= 0, finite)
 *   C       [S][n_L]      spec rows; the property C f(x) >= 0 is merged into the last layer
 *   split   [B][n_relu]   int8 per neuron: +1 enforces h >= 0 (ReLU = identity), -1 enforces
 *                         h < 0 (ReLU = 0), 0 leaves it free; NULL = no splits
 *   alpha   [B][n_relu]   lower slopes of unstable neurons in [0,1] (Eq. 5); NULL = use the
 *                         upper slope u/(u-l) of each neuron's own bounds
 *   lb      [B][S]        out: lb[b][s] <= min_{x in box} (C f_b(x))_s, f_b = the network
 *                         under sub-domain b's splits
 *   l_out, u_out [B][n_relu] optional out: intermediate pre-activation bounds (layer-1 bounds
 *                         are exact; split neurons report their bounds before the split)
 *   code_out [B][n_relu]  optional out: the case of Eq. 5 / Sec. 3.1 each neuron's relaxation
 *                         took, checked in this order: 1 split active (split +1), 2 split
 *                         inactive (split -1), 3 inactive (u <= 0), 4 active (l >= 0),
 *                         5 unstable (l < 0 < u)
 * Intermediate bounds of every layer are recomputed per sub-domain under its own splits. */
int lirpa_bound(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                const int8_t* split, const float* alpha, float* lb, float* l_out, float* u_out,
                int8_t* code_out, void* ws, size_t ws_bytes, hipStream_t stream);

/* lirpa_bound for sub-domains split from a parent whose intermediate bounds are known: every
 * layer's bounds l, u of a sub-domain are intersected with its parent's before the layer is
 * relaxed, l = max(l, l_parent), u = min(u, u_parent).  The paper is silent on reusing them
 * (Sec. 3.1 split constraints, Eq. 9); the reading taken is that a child is a subset of its
 * parent, so the parent's bounds hold on it.  The bound then holds over the sub-domain itself
 * (the box under its split constraints) rather than over the whole box of the split network.
 * Sub-domain b's parent bounds are row b of l_parent, u_parent [B][n_relu] (fp32; e.g. the
 * l_out, u_out of the call that bounded the parent); l_out, u_out report the intersected
 * bounds.  Other arguments as in lirpa_bound (workspace mode 0). */
int lirpa_bound_child(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                      const int8_t* split, const float* alpha, const float* l_parent,
                      const float* u_parent, float* lb, float* l_out, float* u_out,
                      int8_t* code_out, void* ws, size_t ws_bytes, hipStream_t stream);

/* lirpa_bound for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same computation and outputs, with
 * no workspace argument.  Its workspace is the library's own scratch array of 128 MiB per
 * device (a static device array, held from the time the library is loaded on the device until
 * the process ends); the call allocates and frees nothing.  A batch whose workspace exceeds it
 * runs in chunks of as many sub-domains as fit (results are identical to any other chunking).
 * LIRPA_ENOMEM when one sub-domain alone needs more than 128 MiB.  Every call on a device
 * shares that device's array and leaves its contents behind: calls that overlap on one device
 * (from several streams or threads) race and give undefined results. */
int lirpa_bound_noalloc(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                        const int8_t* split, const float* alpha, float* lb, float* l_out,
                        float* u_out, int8_t* code_out, hipStream_t stream);

/* Lower AND upper bounds of the spec rows, the pair (f_lo, f_hi) of Eq. 8 that Algorithm 1's
 * bounding step returns for every sub-domain:
 *   lb[b][s] <= min_{x in box} (C f_b(x))_s   and   ub[b][s] >= max_{x in box} (C f_b(x))_s,
 * ub being max_x of the upper linear function U, computed as -(the lower bound of the rows -C).
 * The intermediate passes (and their l, u, codes) are those of lirpa_bound and are shared by
 * both sides; the final pass bounds the 2S rows [C; -C].  alpha (optional) is the lower slope of
 * both sides.  Arguments as in lirpa_bound; lb, ub [B][S] out; workspace mode 2. */
int lirpa_bound_ul(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                   const int8_t* split, const float* alpha, float* lb, float* ub, float* l_out,
                   float* u_out, int8_t* code_out, void* ws, size_t ws_bytes,
                   hipStream_t stream);

/* As lirpa_bound, plus grad[b][:] = d(sum_s lb[b][s]) / d alpha[b][:] (alpha required).
 * full != 0 differentiates through the recomputed intermediate bounds (Sec. 3.1: they depend on
 * the alphas of earlier layers); full == 0 holds them fixed.  Split and stable neurons get
 * exactly 0. */
int lirpa_bound_grad(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                     const int8_t* split, const float* alpha, int full, float* lb, float* grad,
                     void* ws, size_t ws_bytes, hipStream_t stream);

typedef struct {
  int steps;      /* number of Adam updates (>= 0)                       */
  float lr;       /* step size                                           */
  float beta1;    /* first-moment decay, in [0,1)                        */
  float beta2;    /* second-moment decay, in [0,1)                       */
  float eps_adam; /* denominator guard, > 0                              */
  int t0;         /* updates already taken (bias correction on resume)   */
  int fresh;      /* 1: start from scratch -- the library sets alpha to the upper slope
                     u/(u-l) of each unstable neuron of a heuristic bound pass (1 for
                     active, 0 for inactive neurons), zeroes adam_m and adam_v and takes
                     t0 = 0; 0: continue from the caller's alpha, m, v and t0          */
} lirpa_opt_params;

/* Optimised bounds (Sec. 3.1, Eq. 9 read as a maximisation over alpha): projected Adam ascent
 * on J_b = sum_s lb[b][s], alpha clipped to [0,1] after each step, intermediate bounds
 * recomputed at every iterate.  alpha, adam_m, adam_v [B][n_relu] are in/out (the caller
 * initialises them; m = v = 0 and t0 = 0 for a fresh start).  lb_best [B][S] is out: the
 * elementwise maximum of lb over the steps+1 iterates (each a sound bound).  lb_trace
 * ([steps+1][B][S], optional) receives every iterate's lb. */
int lirpa_optimize(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                   const int8_t* split, float* alpha, float* adam_m, float* adam_v,
                   const lirpa_opt_params* params, float* lb_best, float* lb_trace, void* ws,
                   size_t ws_bytes, hipStream_t stream);

/* Optimised lower AND upper bounds (Eq. 9, each side read as the tightest sound bound: f_lo =
 * max over alpha of min_x L, f_hi = min over alpha of max_x U).  The two sides are optimised
 * with separate slopes, as the intermediate bounds depend on them: alpha_lo, m_lo, v_lo drive
 * lb_best exactly as lirpa_optimize does for C; alpha_up, m_up, v_up drive ub_best, which is
 * -(lirpa_optimize's lb_best for the rows -C).  All [B][n_relu] in/out, lb_best and ub_best
 * [B][S] out; params as in lirpa_optimize (shared by both sides); workspace mode 3. */
int lirpa_optimize_ul(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                      const int8_t* split, float* alpha_lo, float* m_lo, float* v_lo,
                      float* alpha_up, float* m_up, float* v_up, const lirpa_opt_params* params,
                      float* lb_best, float* ub_best, void* ws, size_t ws_bytes,
                      hipStream_t stream);

/* Branch and bound over sub-domains (Algorithm 1, Sec. 3.3-3.4) with the bounding steps above
 * and without its LP fallback: for the single property c^T f(x) >= 0 over the box,
 *   line 2   optimised LiRPA at the root (root_steps Adam steps; 0 = the heuristic slopes);
 *   line 5   batch_pick_out: the `batch` unverified sub-domains with the lowest f_lo (ties: the
 *            earlier record) leave the set P;
 *   line 6   batch_split: each is split on one unstable, unsplit ReLU neuron into a child with it
 *            forced active (+1) and one forced inactive (-1);
 *   line 7   the 2 batch children are bounded in one batch, each from its parent's slopes
 *            (`steps` Adam steps; f_hi at the slopes the lower side ends with);
 *   line 8   Domain_Filter drops the children with f_lo >= 0 (verified), the others join P;
 *   lines 9-10  f_lo, f_hi = the minima over P.
 * The neuron to split is chosen by a stand-in rule (BaBSR's score is not given in the paper):
 * the largest intercept -l u / (u - l) of the upper relaxation line of Eq. 5 under the
 * sub-domain's own bounds, the lowest flat index on ties.  The set P lives in the workspace;
 * the loop reads a small summary from the device once per iteration, so this call synchronises
 * `stream` and returns when the search has ended:
 *   LIRPA_BAB_VERIFIED        P is empty: every sub-domain has f_lo >= 0 (the property holds);
 *   LIRPA_BAB_VIOLATED        a sub-domain's f_hi < 0 (Algorithm 1's loop condition: every point
 *                             of it violates the property, if its splits are feasible -- the
 *                             check the paper leaves to LP);
 *   LIRPA_BAB_UNKNOWN_STUCK   a picked sub-domain has no unstable neuron left to split;
 *   LIRPA_BAB_UNKNOWN_LIMIT   P outgrew max_domains (the paper's eta) or max_iters were run;
 * the last two are where the paper switches to LP.  c is [n_L] on the device. */
typedef enum {
  LIRPA_BAB_VERIFIED = 1,
  LIRPA_BAB_VIOLATED = 2,
  LIRPA_BAB_UNKNOWN_STUCK = 3,
  LIRPA_BAB_UNKNOWN_LIMIT = 4
} lirpa_bab_status;

typedef struct {
  int batch;        /* n of Algorithm 1: sub-domains picked per iteration, 1..1024      */
  int max_domains;  /* eta: largest |P| before stopping; max_domains + batch <= 16384   */
  int max_iters;    /* iteration limit, >= 0                                            */
  int root_steps;   /* Adam steps at the root (the paper takes 100)                     */
  int steps;        /* Adam steps for every new sub-domain (the paper takes 10)         */
  float lr, beta1, beta2, eps_adam; /* as in lirpa_opt_params                           */
} lirpa_bab_params;

typedef struct {
  int status;               /* a lirpa_bab_status                                         */
  float f_lo, f_hi;         /* global bounds at exit: the minima over P (over the verified  */
                            /* sub-domains when P is empty)                                 */
  int iterations;           /* loop iterations run                                          */
  int64_t domains_bounded;  /* sub-domains bounded, the root included                       */
  int domains_left;         /* |P| at exit                                                  */
} lirpa_bab_result;

/* Workspace bytes of lirpa_bab (0 for invalid arguments, SIZE_MAX as in
 * lirpa_workspace_bytes). */
size_t lirpa_bab_workspace_bytes(const lirpa_net* net, const lirpa_bab_params* params);

int lirpa_bab(lirpa_net* net, const float* x0, float eps, const float* c,
              const lirpa_bab_params* params, lirpa_bab_result* result, void* ws,
              size_t ws_bytes, hipStream_t stream);

/* Kernel timing, for profiling harnesses.  Between lirpa_timing_begin() and
 * lirpa_timing_end() every kernel the calls of this thread enqueue is bracketed by a pair of
 * hipEvents recorded on the call's own stream.  lirpa_timing_end() waits for those events and
 * fills up to max_entries records, one per kernel class (summed over its launches), returning
 * the number of classes in *n.  Timing adds two event records per launch. */
typedef struct {
  char name[48];     /* kernel class, e.g. "convT_bound" */
  double total_ms;   /* summed event-to-event time of its launches */
  int64_t launches;
} lirpa_kernel_time;

int lirpa_timing_begin(void);
int lirpa_timing_end(lirpa_kernel_time* out, int max_entries, int* n);

/* Message of the last failed call on this thread ("" if none). */
const char* lirpa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LIRPA_H_ */
