/*
 * ORACLE -- test infrastructure only.
 *
 * Plain, slow, fp64 CPU implementation of batched backward-mode linear relaxation based
 * perturbation analysis (LiRPA / CROWN) with per-sub-domain ReLU split constraints, optional
 * free lower slopes alpha, the analytic gradient of the bound with respect to alpha and the
 * projected Adam loop that optimises them.  It follows Xu et al., "Fast and Complete"
 * (ICLR 2021): Sec. 2.1 (network and problem), Sec. 2.3 Eq. 2-7 (backward bound propagation
 * and the ReLU relaxation of Eq. 5), Sec. 3.1 Eq. 8 (concretisation by Hoelder's inequality),
 * Eq. 9 (optimised bounds; read as a maximisation over alpha) and the split constraints of
 * Sec. 3.1 ("ReLU Split Constraints").
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may load this library.
 * It shares no code, header or table with the GPU library.  All arithmetic is double; fp32
 * inputs are up-cast exactly.  Nothing here is blocked, fused or reordered beyond what the
 * definitions state, so that each function can be read against the paper.
 *
 * Pins (tests/test_oracle_*.py): layer-1 bounds against box-vertex brute force; the transpose
 * of every affine layer against the adjoint identity and an independent convolution;
 * all-split and all-stable exactness against a closed form built forward; the one-neuron
 * triangle closed form; the Appendix A.1 counter-example; sampling soundness; the
 * alpha = LP-dual equivalence on one-hidden-layer nets; finite differences of the gradient;
 * a textbook Adam replay.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* One affine layer T_m: h = W g + b.  ReLU follows every layer except the last (Sec. 2.1). */
typedef struct {
  int kind; /* 0 = fully connected, 1 = 2-D convolution (cross-correlation, zero padding) */
  int in_c, in_h, in_w;
  int out_c, out_h, out_w;
  int k, stride, pad;
  const float* W; /* FC: [out_c][in_c];  conv: [out_c][in_c][k][k] */
  const float* b; /* [out_c]; a conv bias is shared by every position of its channel */
} ref_layer;

enum { REF_OK = 0, REF_EINVAL = -1, REF_ENOMEM = -2 };

/* Stability codes of a ReLU neuron in one sub-domain (oracle step 2). */
enum { ST_SPLIT_ACTIVE = 1, ST_SPLIT_INACTIVE = 2, ST_INACTIVE = 3, ST_ACTIVE = 4, ST_UNSTABLE = 5 };

static long n_in(const ref_layer* t) { return (long)t->in_c * t->in_h * t->in_w; }
static long n_out(const ref_layer* t) { return (long)t->out_c * t->out_h * t->out_w; }

/* ------------------------------------------------------------------------------------------ */
/* The affine map and its transpose.                                                          */
/* ------------------------------------------------------------------------------------------ */

/* h = W g + b (Sec. 2.1, h^(i) = W^(i) g^(i-1), with the bias kept). */
static void affine_fwd(const ref_layer* t, const double* g, double* h) {
  if (t->kind == 0) {
    for (int o = 0; o < t->out_c; ++o) {
      double s = t->b[o];
      for (int i = 0; i < t->in_c; ++i) s += (double)t->W[(long)o * t->in_c + i] * g[i];
      h[o] = s;
    }
    return;
  }
  for (int co = 0; co < t->out_c; ++co)
    for (int yo = 0; yo < t->out_h; ++yo)
      for (int xo = 0; xo < t->out_w; ++xo) {
        double s = t->b[co];
        for (int ci = 0; ci < t->in_c; ++ci)
          for (int ky = 0; ky < t->k; ++ky)
            for (int kx = 0; kx < t->k; ++kx) {
              int yi = yo * t->stride - t->pad + ky, xi = xo * t->stride - t->pad + kx;
              if (yi < 0 || yi >= t->in_h || xi < 0 || xi >= t->in_w) continue;
              s += (double)t->W[(((long)co * t->in_c + ci) * t->k + ky) * t->k + kx] *
                   g[((long)ci * t->in_h + yi) * t->in_w + xi];
            }
        h[((long)co * t->out_h + yo) * t->out_w + xo] = s;
      }
}

/* Coefficient row over the layer's output -> the same linear function over its input:
 * a_in = a_out W (Eq. 4: the backward step through a linear layer).  For a convolution this is
 * the transposed convolution, written as the scatter of each output coefficient over the
 * input positions its forward window reads -- the same index map as affine_fwd. */
static void affine_T(const ref_layer* t, const double* a_out, double* a_in) {
  memset(a_in, 0, sizeof(double) * n_in(t));
  if (t->kind == 0) {
    for (int o = 0; o < t->out_c; ++o) {
      double a = a_out[o];
      if (a == 0.0) continue;
      for (int i = 0; i < t->in_c; ++i) a_in[i] += a * (double)t->W[(long)o * t->in_c + i];
    }
    return;
  }
  for (int co = 0; co < t->out_c; ++co)
    for (int yo = 0; yo < t->out_h; ++yo)
      for (int xo = 0; xo < t->out_w; ++xo) {
        double a = a_out[((long)co * t->out_h + yo) * t->out_w + xo];
        if (a == 0.0) continue;
        for (int ci = 0; ci < t->in_c; ++ci)
          for (int ky = 0; ky < t->k; ++ky)
            for (int kx = 0; kx < t->k; ++kx) {
              int yi = yo * t->stride - t->pad + ky, xi = xo * t->stride - t->pad + kx;
              if (yi < 0 || yi >= t->in_h || xi < 0 || xi >= t->in_w) continue;
              a_in[((long)ci * t->in_h + yi) * t->in_w + xi] +=
                  a * (double)t->W[(((long)co * t->in_c + ci) * t->k + ky) * t->k + kx];
            }
      }
}

/* a . b for a coefficient row a over the layer's output (the bias part of Eq. 6). */
static double bias_dot(const ref_layer* t, const double* a) {
  double s = 0.0;
  long hw = (long)t->out_h * t->out_w;
  for (int c = 0; c < t->out_c; ++c)
    for (long p = 0; p < hw; ++p) s += a[c * hw + p] * (double)t->b[c];
  return s;
}

/* ------------------------------------------------------------------------------------------ */
/* The ReLU relaxation (Eq. 5) with split constraints (Sec. 3.1).                             */
/* ------------------------------------------------------------------------------------------ */

/* Lower line a_lo*h (intercept 0) and upper line a_up*h + b_up of ReLU on [l, u].
 * Cases are checked in this order: split active (the ReLU is forced to the identity), split
 * inactive (forced to zero), always inactive u <= 0, always active l >= 0, unstable.  In the
 * unstable case the upper line is the chord u/(u-l) (h - l); the lower slope is the free
 * alpha when one is given, else the upper slope (the fixed heuristic used without
 * optimisation). */
static int relax(double l, double u, int split, int has_alpha, double alpha, double* a_lo,
                 double* a_up, double* b_up) {
  if (split > 0) { *a_lo = 1.0; *a_up = 1.0; *b_up = 0.0; return ST_SPLIT_ACTIVE; }
  if (split < 0) { *a_lo = 0.0; *a_up = 0.0; *b_up = 0.0; return ST_SPLIT_INACTIVE; }
  if (u <= 0.0) { *a_lo = 0.0; *a_up = 0.0; *b_up = 0.0; return ST_INACTIVE; }
  if (l >= 0.0) { *a_lo = 1.0; *a_up = 1.0; *b_up = 0.0; return ST_ACTIVE; }
  *a_up = u / (u - l);
  *b_up = -u * l / (u - l);
  *a_lo = has_alpha ? alpha : *a_up;
  return ST_UNSTABLE;
}

/* ------------------------------------------------------------------------------------------ */
/* Network bookkeeping.                                                                        */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
  const ref_layer* T; /* T[0..L-1] are the layers T_1..T_L */
  int L;
  long n[64];         /* n[0] = input size, n[m] = size of h^(m) */
  long off[64];       /* offset of ReLU layer m (1..L-1) in the concatenated per-neuron arrays */
  long n_relu, n_max;
} netinfo;

static int net_info(const ref_layer* T, int L, netinfo* ni) {
  if (!T || L < 1 || L > 62) return REF_EINVAL;
  ni->T = T;
  ni->L = L;
  ni->n[0] = n_in(&T[0]);
  ni->n_max = ni->n[0];
  ni->n_relu = 0;
  for (int m = 1; m <= L; ++m) {
    const ref_layer* t = &T[m - 1];
    if (t->kind == 0) {
      if (t->in_h != 1 || t->in_w != 1 || t->out_h != 1 || t->out_w != 1) return REF_EINVAL;
    } else if (t->kind == 1) {
      if (t->k < 1 || t->stride < 1 || t->pad < 0) return REF_EINVAL;
      if (t->out_h != (t->in_h + 2 * t->pad - t->k) / t->stride + 1) return REF_EINVAL;
      if (t->out_w != (t->in_w + 2 * t->pad - t->k) / t->stride + 1) return REF_EINVAL;
    } else {
      return REF_EINVAL;
    }
    if (m > 1 && n_in(t) != ni->n[m - 1]) return REF_EINVAL;
    ni->n[m] = n_out(t);
    if (ni->n[m] > ni->n_max) ni->n_max = ni->n[m];
    if (m < L) { ni->off[m] = ni->n_relu; ni->n_relu += ni->n[m]; }
  }
  return REF_OK;
}

/* Relaxation parameters of one sub-domain for every ReLU neuron. */
typedef struct {
  double *l, *u;             /* intermediate pre-activation bounds, [n_relu] */
  double *a_lo, *a_up, *b_up;
  signed char* code;
} relaxset;

static int relaxset_alloc(relaxset* r, long n) {
  r->l = calloc(n ? n : 1, sizeof(double));
  r->u = calloc(n ? n : 1, sizeof(double));
  r->a_lo = calloc(n ? n : 1, sizeof(double));
  r->a_up = calloc(n ? n : 1, sizeof(double));
  r->b_up = calloc(n ? n : 1, sizeof(double));
  r->code = calloc(n ? n : 1, 1);
  return (r->l && r->u && r->a_lo && r->a_up && r->b_up && r->code) ? REF_OK : REF_ENOMEM;
}
static void relaxset_free(relaxset* r) {
  free(r->l); free(r->u); free(r->a_lo); free(r->a_up); free(r->b_up); free(r->code);
}

/* Fill the relaxation of ReLU layer m from its l, u (already stored in r). */
static void relax_layer(const netinfo* ni, int m, const int8_t* split, const float* alpha,
                        relaxset* r) {
  long o = ni->off[m];
  for (long j = 0; j < ni->n[m]; ++j)
    r->code[o + j] = (signed char)relax(r->l[o + j], r->u[o + j], split ? split[o + j] : 0,
                                        alpha != NULL, alpha ? (double)alpha[o + j] : 0.0,
                                        &r->a_lo[o + j], &r->a_up[o + j], &r->b_up[o + j]);
}

/* ------------------------------------------------------------------------------------------ */
/* Backward bound propagation of one row (Eq. 3-7) and its concretisation (Eq. 8).            */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
  double *A, *B; /* two rows of n_max doubles */
} rowbuf;

/* Lower bound over the box of lam . h^(k) for one sub-domain.  lam has n[k] entries.
 * Starting from the identity at h^(k) (Eq. 3) the row is carried through T_k (Eq. 4), then for
 * m = k-1 .. 1 through the relaxation of ReLU layer m -- non-negative coefficients take the
 * lower line, negative ones the upper line and its intercept (Eq. 6) -- and through T_m.
 * The resulting linear function A x + beta of the input (Eq. 7) is minimised over
 * ||x - x0||_inf <= eps in closed form: A x0 - eps ||A||_1 + beta (Eq. 8).
 * tape (optional): tape[m] receives the coefficient row over g^(m) before the relaxation of
 * layer m.  a_x (optional) receives A; beta_out (optional) receives beta. */
static double bound_row(const netinfo* ni, int k, const double* lam, const relaxset* r,
                        const double* x0, double eps, rowbuf* w, double** tape, double* a_x,
                        double* beta_out) {
  const ref_layer* T = ni->T;
  double beta = bias_dot(&T[k - 1], lam);
  affine_T(&T[k - 1], lam, w->A); /* coefficients over g^(k-1) */
  for (int m = k - 1; m >= 1; --m) {
    long o = ni->off[m];
    double* A = w->A;
    if (tape) memcpy(tape[m], A, sizeof(double) * ni->n[m]);
    for (long j = 0; j < ni->n[m]; ++j) {
      double a = A[j];
      if (a >= 0.0) {
        A[j] = a * r->a_lo[o + j];
      } else {
        beta += a * r->b_up[o + j];
        A[j] = a * r->a_up[o + j];
      }
    }
    beta += bias_dot(&T[m - 1], A);
    affine_T(&T[m - 1], A, w->B);
    double* t = w->A; w->A = w->B; w->B = t;
  }
  double lin = 0.0, l1 = 0.0;
  for (long i = 0; i < ni->n[0]; ++i) {
    lin += w->A[i] * x0[i];
    l1 += fabs(w->A[i]);
  }
  if (a_x) memcpy(a_x, w->A, sizeof(double) * ni->n[0]);
  if (beta_out) *beta_out = beta;
  return lin - eps * l1 + beta;
}

static int rowbuf_alloc(rowbuf* w, long n) {
  w->A = malloc(sizeof(double) * n);
  w->B = malloc(sizeof(double) * n);
  return (w->A && w->B) ? REF_OK : REF_ENOMEM;
}
static void rowbuf_free(rowbuf* w) { free(w->A); free(w->B); }

/* ------------------------------------------------------------------------------------------ */
/* Bounds for a batch of sub-domains.                                                          */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
  netinfo ni;
  const double* x0;
  double eps;
  const float* C;
  int S, B;
  const int8_t* split; /* [B][n_relu] or NULL */
  const float* alpha;  /* [B][n_relu] or NULL */
  /* [B][n_relu] or NULL: intermediate bounds of each sub-domain's parent, intersected with its
   * own (the paper is silent on reusing them; this is the reading that a parent's bounds hold
   * on its children, which are subsets of it) */
  const float* l_par;
  const float* u_par;
  relaxset* rs;        /* [B] */
} problem;

/* Intermediate bounds of every layer, then the relaxation of every layer, for all sub-domains
 * (oracle steps 1, 2, 4).  Pass k bounds h^(k) with the rows +e_j (giving l_j) and -e_j
 * (giving -u_j).  Layer 1 has no relaxation in front of it, so its bounds are exact and the
 * same for every sub-domain. */
static int compute_relaxations(problem* p) {
  const netinfo* ni = &p->ni;
  int err = REF_OK;
  for (int k = 1; k <= ni->L - 1; ++k) {
    long nk = ni->n[k], o = ni->off[k];
    long items = (k == 1) ? 2 * nk : (long)p->B * 2 * nk;
#pragma omp parallel
    {
      rowbuf w = {NULL, NULL};
      double* lam = calloc(nk, sizeof(double));
      int ok = (rowbuf_alloc(&w, ni->n_max) == REF_OK) && lam;
      if (!ok) {
#pragma omp atomic write
        err = REF_ENOMEM;
      }
#pragma omp for schedule(dynamic, 16)
      for (long it = 0; it < items; ++it) {
        if (!ok) continue;
        long b = (k == 1) ? 0 : it / (2 * nk);
        long q = it % (2 * nk);
        long j = q % nk;
        int neg = q >= nk;
        lam[j] = neg ? -1.0 : 1.0;
        double v = bound_row(ni, k, lam, &p->rs[b], p->x0, p->eps, &w, NULL, NULL, NULL);
        lam[j] = 0.0;
        if (neg) p->rs[b].u[o + j] = -v; else p->rs[b].l[o + j] = v;
      }
      free(lam);
      rowbuf_free(&w);
    }
    if (err) return err;
    if (k == 1)
      for (int b = 1; b < p->B; ++b) {
        memcpy(p->rs[b].l + o, p->rs[0].l + o, sizeof(double) * nk);
        memcpy(p->rs[b].u + o, p->rs[0].u + o, sizeof(double) * nk);
      }
    if (p->l_par)
      for (int b = 0; b < p->B; ++b)
        for (long j = 0; j < nk; ++j) {
          long i = (long)b * ni->n_relu + o + j;
          p->rs[b].l[o + j] = fmax(p->rs[b].l[o + j], (double)p->l_par[i]);
          p->rs[b].u[o + j] = fmin(p->rs[b].u[o + j], (double)p->u_par[i]);
        }
    for (int b = 0; b < p->B; ++b)
      relax_layer(ni, k, p->split ? p->split + (long)b * ni->n_relu : NULL,
                  p->alpha ? p->alpha + (long)b * ni->n_relu : NULL, &p->rs[b]);
  }
  return REF_OK;
}

/* Final pass (oracle step 5): the spec rows C_s over h^(L), i.e. the property merged into the
 * last layer (Sec. 2.1). */
static int final_pass(problem* p, double* lb) {
  const netinfo* ni = &p->ni;
  long nL = ni->n[ni->L];
  long items = (long)p->B * p->S;
  int err = REF_OK;
#pragma omp parallel
  {
    rowbuf w = {NULL, NULL};
    double* lam = malloc(sizeof(double) * nL);
    int ok = (rowbuf_alloc(&w, ni->n_max) == REF_OK) && lam;
    if (!ok) {
#pragma omp atomic write
      err = REF_ENOMEM;
    }
#pragma omp for schedule(dynamic, 1)
    for (long it = 0; it < items; ++it) {
      if (!ok) continue;
      long b = it / p->S, s = it % p->S;
      for (long i = 0; i < nL; ++i) lam[i] = (double)p->C[s * nL + i];
      lb[it] = bound_row(ni, ni->L, lam, &p->rs[b], p->x0, p->eps, &w, NULL, NULL, NULL);
    }
    free(lam);
    rowbuf_free(&w);
  }
  return err;
}

static int problem_init(problem* p, const ref_layer* T, int L, const float* x0, float eps,
                        const float* C, int S, int B, const int8_t* split, const float* alpha,
                        double** x0d_out) {
  int e = net_info(T, L, &p->ni);
  if (e) return e;
  if (!x0 || !C || S < 1 || B < 1 || !(eps >= 0.0f) || !isfinite(eps)) return REF_EINVAL;
  double* x0d = malloc(sizeof(double) * p->ni.n[0]);
  if (!x0d) return REF_ENOMEM;
  for (long i = 0; i < p->ni.n[0]; ++i) x0d[i] = x0[i];
  p->x0 = x0d;
  *x0d_out = x0d;
  p->eps = eps;
  p->C = C;
  p->S = S;
  p->B = B;
  p->split = split;
  p->alpha = alpha;
  p->rs = calloc(B, sizeof(relaxset));
  if (!p->rs) return REF_ENOMEM;
  for (int b = 0; b < B; ++b)
    if (relaxset_alloc(&p->rs[b], p->ni.n_relu)) return REF_ENOMEM;
  return REF_OK;
}

static void problem_free(problem* p, double* x0d) {
  if (p->rs)
    for (int b = 0; b < p->B; ++b) relaxset_free(&p->rs[b]);
  free(p->rs);
  free(x0d);
}

static void set_threads(int nthreads) {
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
}

/* Number of ReLU neurons, sum over layers 1..L-1 of n_m; <0 on an invalid chain. */
long ref_num_relu(const ref_layer* T, int L) {
  netinfo ni;
  int e = net_info(T, L, &ni);
  return e ? e : ni.n_relu;
}

/* lb[b][s] <= min over the box of (C f_b(x))_s for each sub-domain b, where f_b is the network
 * under the split constraints of b.  alpha == NULL selects the heuristic lower slope.
 * l_out, u_out, code_out (optional, [B][n_relu]) receive the intermediate bounds and
 * stability codes. */
static int bound_impl(const ref_layer* T, int L, const float* x0, float eps, const float* C,
                      int S, int B, const int8_t* split, const float* alpha,
                      const float* l_par, const float* u_par, double* lb, double* l_out,
                      double* u_out, signed char* code_out, int nthreads) {
  set_threads(nthreads);
  problem p;
  memset(&p, 0, sizeof p);
  double* x0d = NULL;
  int e = problem_init(&p, T, L, x0, eps, C, S, B, split, alpha, &x0d);
  p.l_par = l_par;
  p.u_par = u_par;
  if (!e) e = compute_relaxations(&p);
  if (!e) e = final_pass(&p, lb);
  if (!e)
    for (int b = 0; b < B; ++b) {
      long n = p.ni.n_relu;
      if (l_out) memcpy(l_out + (long)b * n, p.rs[b].l, sizeof(double) * n);
      if (u_out) memcpy(u_out + (long)b * n, p.rs[b].u, sizeof(double) * n);
      if (code_out) memcpy(code_out + (long)b * n, p.rs[b].code, n);
    }
  problem_free(&p, x0d);
  return e;
}

int ref_bound(const ref_layer* T, int L, const float* x0, float eps, const float* C, int S,
              int B, const int8_t* split, const float* alpha, double* lb, double* l_out,
              double* u_out, signed char* code_out, int nthreads) {
  return bound_impl(T, L, x0, eps, C, S, B, split, alpha, NULL, NULL, lb, l_out, u_out,
                    code_out, nthreads);
}

/* ref_bound with each sub-domain's intermediate bounds intersected, layer by layer before its
 * relaxation, with its parent's l_par, u_par ([B][n_relu], fp32): l = max(l, l_par),
 * u = min(u, u_par).  The result bounds min over the sub-domain itself (not over the box of
 * the split network), and l_out, u_out report the intersected bounds. */
int ref_bound_child(const ref_layer* T, int L, const float* x0, float eps, const float* C,
                    int S, int B, const int8_t* split, const float* alpha, const float* l_par,
                    const float* u_par, double* lb, double* l_out, double* u_out,
                    signed char* code_out, int nthreads) {
  if (!l_par || !u_par) return REF_EINVAL;
  return bound_impl(T, L, x0, eps, C, S, B, split, alpha, l_par, u_par, lb, l_out, u_out,
                    code_out, nthreads);
}

/* The final linear lower-bounding functions L_s(x) = A_s x + beta_s of one sub-domain
 * (Eq. 7), A: [S][n0], beta: [S].  For tests of concretisation and pointwise soundness. */
int ref_linear_bound_fn(const ref_layer* T, int L, const float* x0, float eps, const float* C,
                        int S, const int8_t* split, const float* alpha, double* A, double* beta) {
  problem p;
  memset(&p, 0, sizeof p);
  double* x0d = NULL;
  int e = problem_init(&p, T, L, x0, eps, C, S, 1, split, alpha, &x0d);
  if (!e) e = compute_relaxations(&p);
  if (!e) {
    rowbuf w = {NULL, NULL};
    long nL = p.ni.n[L];
    double* lam = malloc(sizeof(double) * nL);
    if (rowbuf_alloc(&w, p.ni.n_max) || !lam) e = REF_ENOMEM;
    for (int s = 0; !e && s < S; ++s) {
      for (long i = 0; i < nL; ++i) lam[i] = (double)C[(long)s * nL + i];
      bound_row(&p.ni, L, lam, &p.rs[0], p.x0, p.eps, &w, NULL, A + (long)s * p.ni.n[0],
                &beta[s]);
    }
    free(lam);
    rowbuf_free(&w);
  }
  problem_free(&p, x0d);
  return e;
}

/* ------------------------------------------------------------------------------------------ */
/* Gradient of J_b = sum_s lb[b][s] with respect to alpha (Sec. 3.1, Eq. 9).                  */
/* ------------------------------------------------------------------------------------------ */

/* Reverse sweep for one sub-domain.  The bound of a row is L_r(x*) with the witness
 * x* = x0 - eps sign(A_r) (sign(0) = 0), and L_r(x) is the row's linear function evaluated by
 * running x forward through the row's relaxed network: z_0 = x, G_m = T_m z_{m-1}, and
 * z_m = a_lo G_m where the row's coefficient over g^(m) was >= 0, else a_up G_m + b_up.  So
 * dL_r/da_lo = max(A~,0) G, dL_r/da_up = min(A~,0) G and dL_r/db_up = min(A~,0), where A~ is
 * the row's coefficient over g^(m) before the relaxation.  For an unstable, unsplit neuron
 * a_lo = alpha, a_up = u/(u-l) and b_up = -u l/(u-l), which carries the adjoint into the
 * intermediate bounds l, u; those come from earlier passes (l_j from row +e_j, u_j = -lb of row
 * -e_j), so passes are visited in descending order with row weights [g_l ; -g_u].  When
 * full == 0 only the final pass is visited, i.e. the gradient with the intermediate bounds
 * frozen.  Layer-1 bounds do not depend on alpha. */
static int grad_subdomain(const problem* p, int b, int full, double* g_alpha) {
  const netinfo* ni = &p->ni;
  const relaxset* r = &p->rs[b];
  long nr = ni->n_relu, n0 = ni->n[0];
  int L = ni->L;
  double* g_l = calloc(nr ? nr : 1, sizeof(double));
  double* g_u = calloc(nr ? nr : 1, sizeof(double));
  double* tapemem = malloc(sizeof(double) * (nr ? nr : 1));
  double* tape[64];
  double* a_x = malloc(sizeof(double) * n0);
  double* lam = malloc(sizeof(double) * ni->n_max);
  double* z = malloc(sizeof(double) * ni->n_max);
  double* G = malloc(sizeof(double) * ni->n_max);
  rowbuf w = {NULL, NULL};
  int e = (g_l && g_u && tapemem && a_x && lam && z && G) ? REF_OK : REF_ENOMEM;
  if (!e) e = rowbuf_alloc(&w, ni->n_max);
  if (e) goto done;
  for (int m = 1; m < L; ++m) tape[m] = tapemem + ni->off[m];
  memset(g_alpha, 0, sizeof(double) * nr);

  for (int P = L; P >= 2; --P) {
    if (!full && P < L) break;
    long nP = ni->n[P];
    long rows = (P == L) ? p->S : 2 * nP;
    for (long q = 0; q < rows; ++q) {
      double wr;
      memset(lam, 0, sizeof(double) * nP);
      if (P == L) {
        wr = 1.0;
        for (long i = 0; i < nP; ++i) lam[i] = (double)p->C[q * nP + i];
      } else if (q < nP) {
        wr = g_l[ni->off[P] + q];
        lam[q] = 1.0;
      } else {
        wr = -g_u[ni->off[P] + (q - nP)];
        lam[q - nP] = -1.0;
      }
      if (wr == 0.0) continue;
      bound_row(ni, P, lam, r, p->x0, p->eps, &w, tape, a_x, NULL);
      for (long i = 0; i < n0; ++i)
        z[i] = p->x0[i] - p->eps * (a_x[i] > 0.0 ? 1.0 : (a_x[i] < 0.0 ? -1.0 : 0.0));
      for (int m = 1; m <= P - 1; ++m) {
        long o = ni->off[m];
        affine_fwd(&ni->T[m - 1], z, G);
        for (long j = 0; j < ni->n[m]; ++j) {
          double t = tape[m][j], gj = G[j];
          if (r->code[o + j] == ST_UNSTABLE && p->alpha) {
            double lj = r->l[o + j], uj = r->u[o + j], d = uj - lj;
            double tp = t > 0.0 ? t : 0.0, tn = t < 0.0 ? t : 0.0;
            double da = wr * tn * gj, db = wr * tn;
            g_alpha[o + j] += wr * tp * gj;
            g_l[o + j] += da * uj / (d * d) - db * uj * uj / (d * d);
            g_u[o + j] += -da * lj / (d * d) + db * lj * lj / (d * d);
          }
          z[j] = (t >= 0.0) ? r->a_lo[o + j] * gj : r->a_up[o + j] * gj + r->b_up[o + j];
        }
      }
    }
  }
done:
  rowbuf_free(&w);
  free(g_l); free(g_u); free(tapemem); free(a_x); free(lam); free(z); free(G);
  return e;
}

static int grad_all(problem* p, int full, double* grad) {
  int err = REF_OK;
#pragma omp parallel for schedule(dynamic, 1)
  for (int b = 0; b < p->B; ++b) {
    int e = grad_subdomain(p, b, full, grad + (long)b * p->ni.n_relu);
    if (e) {
#pragma omp atomic write
      err = e;
    }
  }
  return err;
}

/* lb as in ref_bound at the given alpha (required), and grad[b][:] = dJ_b/dalpha[b][:] with
 * J_b = sum_s lb[b][s].  full = 1 differentiates through the recomputed intermediate bounds,
 * full = 0 holds them fixed.  Split and stable neurons get exactly 0. */
int ref_bound_grad(const ref_layer* T, int L, const float* x0, float eps, const float* C, int S,
                   int B, const int8_t* split, const float* alpha, int full, double* lb,
                   double* grad, int nthreads) {
  if (!alpha || !grad || !lb) return REF_EINVAL;
  set_threads(nthreads);
  problem p;
  memset(&p, 0, sizeof p);
  double* x0d = NULL;
  int e = problem_init(&p, T, L, x0, eps, C, S, B, split, alpha, &x0d);
  if (!e) e = compute_relaxations(&p);
  if (!e) e = final_pass(&p, lb);
  if (!e) e = grad_all(&p, full, grad);
  problem_free(&p, x0d);
  return e;
}

/* ------------------------------------------------------------------------------------------ */
/* Optimised bounds (Eq. 9 read as max over alpha; Sec. 3.1 projected gradient).             */
/* ------------------------------------------------------------------------------------------ */

/* Projected Adam ascent on J_b(alpha) = sum_s lb[b][s] for every sub-domain, each alpha kept in
 * [0, 1] by clipping after every step; intermediate bounds are recomputed at every iterate.
 * alpha (in/out, [B][n_relu]) starts at the caller's value; m, v (in/out) are the Adam moments
 * and t0 the number of steps already taken (0 for a fresh start).  After `steps` updates,
 * lb_best[b][s] is the elementwise maximum of lb over the steps+1 iterates visited (each one
 * is a sound bound).  lb_trace (optional, [steps+1][B][S]) receives every iterate's lb. */
int ref_optimize(const ref_layer* T, int L, const float* x0, float eps, const float* C, int S,
                 int B, const int8_t* split, double* alpha, double* m, double* v, int steps,
                 double lr, double beta1, double beta2, double eps_adam, int t0, double* lb_best,
                 double* lb_trace, int nthreads) {
  if (!alpha || !m || !v || !lb_best || steps < 0 || t0 < 0) return REF_EINVAL;
  long nr = ref_num_relu(T, L);
  if (nr < 0) return (int)nr;
  long na = (long)B * nr;
  float* af = malloc(sizeof(float) * (na ? na : 1));
  double* g = malloc(sizeof(double) * (na ? na : 1));
  double* lb = malloc(sizeof(double) * (long)B * S);
  int e = (af && g && lb) ? REF_OK : REF_ENOMEM;
  for (int t = 0; !e && t <= steps; ++t) {
    /* The GPU and this oracle both hand alpha to the bound as fp32. */
    for (long i = 0; i < na; ++i) af[i] = (float)alpha[i];
    if (t < steps)
      e = ref_bound_grad(T, L, x0, eps, C, S, B, split, af, 1, lb, g, nthreads);
    else
      e = ref_bound(T, L, x0, eps, C, S, B, split, af, lb, NULL, NULL, NULL, nthreads);
    if (e) break;
    for (long i = 0; i < (long)B * S; ++i) {
      if (t == 0 || lb[i] > lb_best[i]) lb_best[i] = lb[i];
      if (lb_trace) lb_trace[(long)t * B * S + i] = lb[i];
    }
    if (t == steps) break;
    int tt = t0 + t + 1;
    double c1 = 1.0 - pow(beta1, tt), c2 = 1.0 - pow(beta2, tt);
    for (long i = 0; i < na; ++i) {
      m[i] = beta1 * m[i] + (1.0 - beta1) * g[i];
      v[i] = beta2 * v[i] + (1.0 - beta2) * g[i] * g[i];
      double step = lr * (m[i] / c1) / (sqrt(v[i] / c2) + eps_adam);
      double a = alpha[i] + step;
      alpha[i] = a < 0.0 ? 0.0 : (a > 1.0 ? 1.0 : a);
    }
  }
  free(af); free(g); free(lb);
  return e;
}

/* ------------------------------------------------------------------------------------------ */
/* Plain network evaluation, for tests.                                                        */
/* ------------------------------------------------------------------------------------------ */

/* out[i][:] = f(x_i) for N inputs.  split (optional, [n_relu]) replaces split-active ReLUs by
 * the identity and split-inactive ones by zero (the network f_s of a sub-domain). */
int ref_forward(const ref_layer* T, int L, const double* x, long N, const int8_t* split,
                double* out) {
  netinfo ni;
  int e = net_info(T, L, &ni);
  if (e) return e;
#pragma omp parallel
  {
    double* a = malloc(sizeof(double) * ni.n_max);
    double* h = malloc(sizeof(double) * ni.n_max);
#pragma omp for schedule(static)
    for (long i = 0; i < N; ++i) {
      if (!a || !h) continue;
      memcpy(a, x + i * ni.n[0], sizeof(double) * ni.n[0]);
      for (int m = 1; m <= L; ++m) {
        affine_fwd(&T[m - 1], a, h);
        if (m < L)
          for (long j = 0; j < ni.n[m]; ++j) {
            int s = split ? split[ni.off[m] + j] : 0;
            a[j] = s > 0 ? h[j] : (s < 0 ? 0.0 : (h[j] > 0.0 ? h[j] : 0.0));
          }
        else
          memcpy(out + i * ni.n[L], h, sizeof(double) * ni.n[L]);
      }
    }
    free(a);
    free(h);
  }
  return REF_OK;
}

/* Transposed application of one layer to R coefficient rows (for the adjoint-identity pin). */
int ref_layer_T(const ref_layer* t, const double* a_out, long R, double* a_in) {
  for (long r = 0; r < R; ++r) affine_T(t, a_out + r * n_out(t), a_in + r * n_in(t));
  return REF_OK;
}

/* Forward application of one layer to R inputs. */
int ref_layer_fwd(const ref_layer* t, const double* g, long R, double* h) {
  for (long r = 0; r < R; ++r) affine_fwd(t, g + r * n_in(t), h + r * n_out(t));
  return REF_OK;
}

/* The relaxation of Eq. 5 for one neuron, for the unit tests of its case table. */
int ref_relax(double l, double u, int split, int has_alpha, double alpha, double* out3) {
  return relax(l, u, split, has_alpha, alpha, &out3[0], &out3[1], &out3[2]);
}
