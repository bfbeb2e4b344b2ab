// Batched backward-mode LiRPA (CROWN) bounds for gfx950 -- host API and kernels.
//
// Method: Xu et al., "Fast and Complete" (ICLR 2021), Sec. 2.3 Eq. 3-7 (backward propagation
// of the bound matrix through affine layers and the ReLU relaxation of Eq. 5), Sec. 3.1 Eq. 8
// (concretisation by Hoelder's inequality over the l_inf box) and the ReLU split constraints of
// Sec. 3.1.
//
// Data layout.  A "pass" bounds Q = (sub-domains in the chunk) x R rows at once; every bound
// matrix slab is stored [n][Qp] with the row index q = b*R + r fastest (Qp = Q rounded up to
// 64), so one lane owns one row for the whole pass: loads and stores of a slab are coalesced
// across the wave, weights are wave-uniform (scalar loads), and the per-row sums of the
// relaxation (bias accumulation) and of the concretisation need no cross-lane reduction.
//
// Pass structure (one chunk of sub-domains):
//   pass 1       rows +-e_j of h^(1), once per call: exact layer-1 bounds (shared);
//   pass k       rows +-e_j of h^(k), 2 <= k <= L-1: init writes relax_{k-1}(+-W_k rows),
//                then stage m = k-1..1 applies T_m^T with the relaxation of layer m-1 fused in
//                its epilogue, and the last stage concretises into l^(k), u^(k);
//   final pass   spec rows C over h^(L): stage L..1 as above, concretising into lb.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "lirpa.h"

namespace {

// ---------------------------------------------------------------------------------------------
// Errors
// ---------------------------------------------------------------------------------------------
thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

// Kernel timing (lirpa_timing_begin / lirpa_timing_end): event pairs around every launch.
struct TimingRec {
  std::string cls;
  size_t ev;  // index of the first event of the pair in the pool
};
struct TimingState {
  bool on = false;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<TimingRec> recs;
};
thread_local TimingState g_tim;

// Enqueue one kernel through `launch`, bracketed by events when timing is on.
template <typename F>
int launch_k(const std::string& cls, hipStream_t st, F&& launch) {
  size_t ev = 0;
  if (g_tim.on) {
    while (g_tim.pool.size() < g_tim.used + 2) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return fail(LIRPA_EDEVICE, "hipEventCreate failed");
      g_tim.pool.push_back(e);
    }
    ev = g_tim.used;
    g_tim.used += 2;
    if (hipEventRecord(g_tim.pool[ev], st) != hipSuccess)
      return fail(LIRPA_EDEVICE, "hipEventRecord failed");
  }
  launch();
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(LIRPA_EDEVICE, "%s: %s", cls.c_str(), hipGetErrorString(e));
  if (g_tim.on) {
    if (hipEventRecord(g_tim.pool[ev + 1], st) != hipSuccess)
      return fail(LIRPA_EDEVICE, "hipEventRecord failed");
    g_tim.recs.push_back(TimingRec{cls, ev});
  }
  return LIRPA_OK;
}

std::string tag(const char* kind, int m, int k) {
  char b[64];
  snprintf(b, sizeof b, "%s[layer%d,pass%d]", kind, m, k);
  return b;
}

constexpr int kMaxLayers = 32;
constexpr int kBlock = 256;

long n_in_of(const lirpa_layer& t) { return (long)t.in_c * t.in_h * t.in_w; }
long n_out_of(const lirpa_layer& t) { return (long)t.out_c * t.out_h * t.out_w; }
long round_up(long x, long m) { return (x + m - 1) / m * m; }

}  // namespace

// Findings of the check of a call's device inputs (LIRPA_VALIDATE=1), one word per kind: [0] a
// split value outside {-1, 0, 1} (Sec. 3.1 split constraints), [1] an alpha outside [0, 1] or not
// a number (Eq. 5), [2] a non-finite x0, [3] a non-finite spec entry.  Each device holds its own
// copy; a finding is recorded by plain stores of 1 (idempotent, no atomics) and read and cleared
// by the host through the symbol.
static __device__ unsigned int g_check[4];

// Scratch array of lirpa_bound_noalloc, the workspace of callers that cannot allocate device
// memory.  Each device holds its own copy from the time the library is loaded on it until the
// process ends.  Host code never passes the array's name to a kernel or a copy (it is a host-side
// stand-in there): it takes the device address of the current device's copy, looked up once per
// device with hipGetSymbolAddress (scratch_address()).
constexpr size_t kScratchBytes = size_t(128) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct lirpa_net {
  std::vector<lirpa_layer> T;  // T[0..L-1] = T_1..T_L
  int L = 0;
  long n[kMaxLayers + 1] = {};    // n[0] input size, n[m] size of h^(m)
  long off[kMaxLayers + 1] = {};  // offset of ReLU layer m in per-neuron arrays
  long n_relu = 0;
  // internal layout of the relaxation parameters: every layer segment starts on a 16-byte
  // boundary so that rows of a feature map load as float4
  long poff[kMaxLayers + 1] = {};
  long pstride = 0;
};

namespace {

// ---------------------------------------------------------------------------------------------
// Device-side descriptors
// ---------------------------------------------------------------------------------------------
struct DLayer {
  int kind, in_c, in_h, in_w, out_c, out_h, out_w, k, stride, pad;
  const float* W;
  const float* b;
};

DLayer dlayer(const lirpa_layer& t) {
  return DLayer{t.kind, t.in_c, t.in_h, t.in_w, t.out_c, t.out_h, t.out_w,
                t.k,    t.stride, t.pad, t.W,  t.b};
}

enum { MODE_SLAB = 0, MODE_BOUND = 1 };

typedef float float4v __attribute__((ext_vector_type(4)));

// 16-row tile of a block, XCD-aware.  Workgroups are dispatched round-robin over the 8 XCDs,
// each with its own L2, and a 16-row tile covers half of a 128-byte line in every slab row: tiles
// 2k and 2k+1 go to blocks b and b+8, which land on the same XCD, so each line is fetched and
// written back by one L2.  Grids are padded to a multiple of 16 blocks; blocks past the last
// tile exit at once.
__device__ __forceinline__ unsigned xcd_tile(unsigned blk) {
  return (blk & ~15u) + ((blk & 7u) << 1) + ((blk >> 3) & 1u);
}

// Block index of a kernel whose blocks read per-sub-domain data (relaxation parameters): the
// blocks of XCD x (those with blockIdx.x mod 8 == x) take the contiguous range
// [x n/8, (x+1) n/8) in order, n = gridDim.x, so the consecutive blocks of one sub-domain
// fetch its data into one L2 instead of all eight.  Identity when n is not a multiple of 8.
__device__ __forceinline__ unsigned xcd_range(unsigned blk) {
  const unsigned n = gridDim.x;
  return (n & 7u) ? blk : (blk & 7u) * (n >> 3) + (blk >> 3);
}

// Index of the calling wave in its block, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

// Store v at byte offset boff (< 2^31) from the wave-uniform address row: a buffer store with
// the base in scalar registers, so no per-lane 64-bit address arithmetic.
__device__ __forceinline__ void store_row(float* row, unsigned boff, float v) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(row, (short)0, 0x7fffffff, 0x00020000);
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), rs, boff, 0, 0);
}

// Workgroup barrier for LDS traffic only: waits for this wave's LDS operations, not for its
// outstanding global stores (which __syncthreads() would also drain).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Where a stage's output row goes.
//  MODE_SLAB : coefficients over g^(m) are relaxed with layer m's (a_lo, a_up, b_up) of the
//              row's sub-domain (Eq. 6: non-negative entries take the lower line, negative ones
//              the upper line and its intercept), the bias of layer m is dotted in, and the
//              relaxed row is stored in out[i*ldq + q].
//  MODE_BOUND: coefficients over the input x are concretised (Eq. 8):
//              value = A x0 - eps ||A||_1 + beta; row r < n_half goes to lo[b*bstride + r],
//              a row r >= n_half to hi[b*bstride + r - n_half] negated (an upper bound).
//              When x0 is null the linear term is already in beta: with A = A1 W1 (A1 the
//              relaxed coefficients over h^(1)), A x0 + A1 b1 = A1 (W1 x0 + b1), so the
//              relaxation onto layer 1 dots A1 with z1 = W1 x0 + b1 instead of with b1
//              (bias_hw == 1 then means a per-neuron bias vector).
// Sign of a coefficient as stored in the gradient tape over x: -1, 0 or +1.
__device__ __forceinline__ int8_t sign8(float a) {
  return (int8_t)(a > 0.f ? 1 : (a < 0.f ? -1 : 0));
}

struct Sink {
  float* out;
  long ldq;
  const float* a_lo;
  const float* a_up;
  const float* b_up;
  long pstride;  // per-sub-domain stride of the relaxation parameters
  const float* bias;
  int bias_hw;
  const float* x0;
  float eps;
  float* beta;  // running bias of each row, [Qp]
  long R;       // rows per sub-domain
  float* lo;
  float* hi;
  long bstride;
  long n_half;
  float* tape;  // optional: the coefficient before relaxation (relaxing stages), [i*ldq + q]
  // optional (concretising stages): the sign of the coefficient over x, the only part of it
  // the witness x* = x0 - eps sign(A_x) of the gradient needs, one byte per entry [i*ldq + q]
  int8_t* tsign;
};

// Input of the first backward stage of a pass that starts at a fully connected layer k (rows
// +-e_j over h^(k), nk of each sign, R = 2 nk per sub-domain): carried through T_k (Eq. 4) row j
// becomes +-(row j of W_k) over g^(k-1), which is then relaxed with ReLU layer k-1 (Eq. 6).  A
// stage through layer k-1 can build these coefficients as it goes instead of reading them from
// a slab.
struct FcSrc {
  const float* W;     // W_k, [nk][nin] (row j contiguous, 16-byte aligned)
  const float* b;     // b_k, [nk]
  int nk;
  const float* a_lo;  // relaxation of ReLU layer k-1 (per sub-domain, stride Sink::pstride)
  const float* a_up;
  const float* b_up;
  // k_convT_fc_bound only (rows interleaved: row 2j is +e_j, row 2j + 1 is -e_j): the
  // relaxation of layer k it writes from the bounds (as k_relax_params would)
  const int8_t* split;  // per sub-domain, stride n_relu, at the layer's offset off
  const float* alpha;
  float* r_lo;          // per sub-domain, stride Sink::pstride
  float* r_up;
  float* r_bu;
  int8_t* code;         // stride n_relu, at offset off
  long n_relu, off;
  const float* lpar;    // parent bounds (stride n_relu, at offset off) or null
  const float* upar;
  // spec source of k_convT_fc_bound (the final pass from the merged spec rows): b holds
  // C W_L [S][nk] followed by C b_L [S]; r_lo, r_up, r_bu the relaxation of layer L-1 (read);
  // a_lo, a_up, b_up that of layer L-2; the two layers' bias vectors
  const float* sbias_k = nullptr;   // layer L-2
  const float* sbias_k1 = nullptr;  // layer L-1
};

struct Acc {
  float beta, lin, l1;
};

template <int MODE>
__device__ __forceinline__ void sink_put(const Sink& s, Acc& acc, long i, float a, long q,
                                         long b) {
  if constexpr (MODE == MODE_SLAB) {
    if (s.tape) s.tape[i * s.ldq + q] = a;
  } else {
    if (s.tsign) s.tsign[i * s.ldq + q] = sign8(a);
  }
  if constexpr (MODE == MODE_SLAB) {
    long pi = b * s.pstride + i;
    float ah;
    if (a >= 0.f) {
      ah = a * s.a_lo[pi];
    } else {
      acc.beta = fmaf(a, s.b_up[pi], acc.beta);
      ah = a * s.a_up[pi];
    }
    acc.beta = fmaf(ah, s.bias[(unsigned)i / (unsigned)s.bias_hw], acc.beta);
    s.out[i * s.ldq + q] = ah;
  } else {
    if (s.x0) acc.lin = fmaf(a, s.x0[i], acc.lin);
    acc.l1 += fabsf(a);
  }
}

// use_beta: add the row's running bias kept in s.beta (stages after an init).
template <int MODE>
__device__ __forceinline__ void sink_finish(const Sink& s, const Acc& acc, long q, long b, long r,
                                            bool first) {
  if constexpr (MODE == MODE_SLAB) {
    s.beta[q] = first ? acc.beta : s.beta[q] + acc.beta;
  } else {
    float beta = first ? acc.beta : s.beta[q] + acc.beta;
    float v = acc.lin - s.eps * acc.l1 + beta;
    if (r < s.n_half)
      s.lo[b * s.bstride + r] = v;
    else
      s.hi[b * s.bstride + (r - s.n_half)] = -v;
  }
}

// Relaxation of one ReLU neuron with bounds l <= u (Eq. 5 with the split override of Sec. 3.1,
// checked in the order: split, u <= 0, l >= 0, unstable): lower slope a_lo (alpha when given,
// else the upper slope), upper line a_up x + b_up, and the stability code (1 split active,
// 2 split inactive, 3 inactive, 4 active, 5 unstable).
struct Relax1 {
  float lo, up, bu;
  int code;
};

__device__ __forceinline__ Relax1 relax_neuron(float l, float u, int sp, const float* alpha) {
  if (sp > 0) return {1.f, 1.f, 0.f, 1};
  if (sp < 0) return {0.f, 0.f, 0.f, 2};
  if (u <= 0.f) return {0.f, 0.f, 0.f, 3};
  if (l >= 0.f) return {1.f, 1.f, 0.f, 4};
  const float d = u - l;
  const float up = u / d;
  return {alpha ? *alpha : up, up, -(u * l) / d, 5};
}

// A sub-domain's bounds of one neuron intersected with its parent's (lp, up at index i, both
// null when no parent bounds are given): a child is a subset of its parent, so the parent's
// bounds hold on it.
__device__ __forceinline__ void parent_clip(float& l, float& u, const float* lp, const float* up,
                                            long i) {
  if (lp) {
    l = fmaxf(l, lp[i]);
    u = fminf(u, up[i]);
  }
}

// ---------------------------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------------------------

// Rows +-e_j over h^(k) (j = r mod n_k, sign + for r < n_k): carried through T_k (Eq. 4) they
// become +-(row j of W_k) over g^(k-1), with bias +-b_k[j].
// WT (optional, LINEAR only): the weights transposed, [in_c][out_c], so that the lanes of a
// wave (consecutive j) read consecutive addresses.
template <int MODE>
__device__ __forceinline__ void init_row(const DLayer& t, const float* __restrict__ WT,
                                         const Sink& s, long q) {
  long b = q / s.R, r = q % s.R;
  long nk = (long)t.out_c * t.out_h * t.out_w;
  long j = r % nk;
  float sgn = r < nk ? 1.f : -1.f;
  int hw = t.out_h * t.out_w;
  Acc acc{sgn * t.b[j / hw], 0.f, 0.f};
  if (t.kind == LIRPA_LINEAR) {
    if (WT)
      for (int i = 0; i < t.in_c; ++i)
        sink_put<MODE>(s, acc, i, sgn * WT[(long)i * t.out_c + j], q, b);
    else
      for (int i = 0; i < t.in_c; ++i)
        sink_put<MODE>(s, acc, i, sgn * t.W[j * t.in_c + i], q, b);
  } else if (MODE == MODE_BOUND) {
    // concretising: only the kernel window contributes
    int co = (int)(j / hw), yo = (int)((j / t.out_w) % t.out_h), xo = (int)(j % t.out_w);
    int y0 = yo * t.stride - t.pad, x0 = xo * t.stride - t.pad;
    for (int ci = 0; ci < t.in_c; ++ci)
      for (int ky = 0; ky < t.k; ++ky) {
        int yi = y0 + ky;
        if (yi < 0 || yi >= t.in_h) continue;
        for (int kx = 0; kx < t.k; ++kx) {
          int xi = x0 + kx;
          if (xi < 0 || xi >= t.in_w) continue;
          float a = sgn * t.W[(((long)co * t.in_c + ci) * t.k + ky) * t.k + kx];
          sink_put<MODE>(s, acc, ((long)ci * t.in_h + yi) * t.in_w + xi, a, q, b);
        }
      }
  } else {
    int co = (int)(j / hw), yo = (int)((j / t.out_w) % t.out_h), xo = (int)(j % t.out_w);
    int y0 = yo * t.stride - t.pad, x0 = xo * t.stride - t.pad;
    for (int ci = 0; ci < t.in_c; ++ci)
      for (int yi = 0; yi < t.in_h; ++yi)
        for (int xi = 0; xi < t.in_w; ++xi) {
          int ky = yi - y0, kx = xi - x0;
          float a = 0.f;
          if (ky >= 0 && ky < t.k && kx >= 0 && kx < t.k)
            a = sgn * t.W[(((long)co * t.in_c + ci) * t.k + ky) * t.k + kx];
          sink_put<MODE>(s, acc, ((long)ci * t.in_h + yi) * t.in_w + xi, a, q, b);
        }
  }
  sink_finish<MODE>(s, acc, q, b, r, true);
}

template <int MODE>
__global__ void __launch_bounds__(kBlock) k_init_rows(DLayer t, const float* __restrict__ WT,
                                                      long Q, Sink s) {
  long q = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (q >= Q) return;
  init_row<MODE>(t, WT, s, q);
}

// Pass initialisation for the rows +-e_j of a fully connected layer k, relaxed onto ReLU layer
// k-1 (slab sink).  Block: 64 rows x 4 waves; each wave covers a quarter of the coefficients
// (float4 parameter loads), and the rows' bias terms are summed through LDS in a fixed order.
__global__ void __launch_bounds__(256) k_init_fc_rows(DLayer t, const float* __restrict__ WT,
                                                      long Q, Sink s) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, w = wave_id();
  const long q = blockIdx.x * 64L + lane;
  const bool ok = q < Q;
  const long qq = ok ? q : 0;
  const long b = qq / s.R, r = qq % s.R;
  const int nk = t.out_c, nin = t.in_c;
  const int j = (int)(r % nk);
  const float sgn = r < nk ? 1.f : -1.f;
  const int chunk = ((nin + 15) / 16) * 4;
  const int i0 = w * chunk, i1 = min(nin, i0 + chunk);
  const long pb = b * s.pstride;
  const unsigned hw = (unsigned)s.bias_hw;
  float beta = 0.f;
  if (ok) {
    int i = i0;
    for (; i + 4 <= i1; i += 4) {
      const float4v lo = *reinterpret_cast<const float4v*>(s.a_lo + pb + i);
      const float4v up = *reinterpret_cast<const float4v*>(s.a_up + pb + i);
      const float4v bu = *reinterpret_cast<const float4v*>(s.b_up + pb + i);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float a = sgn * WT[(long)(i + u) * nk + j];
        const long idx = (long)(i + u) * s.ldq + q;
        if (s.tape) s.tape[idx] = a;
        const float ah = a >= 0.f ? a * lo[u] : a * up[u];
        beta = fmaf(fminf(a, 0.f), bu[u], beta);
        beta = fmaf(ah, s.bias[(unsigned)(i + u) / hw], beta);
        s.out[idx] = ah;
      }
    }
    for (; i < i1; ++i) {
      const float a = sgn * WT[(long)i * nk + j];
      const long idx = (long)i * s.ldq + q;
      if (s.tape) s.tape[idx] = a;
      const float ah = a >= 0.f ? a * s.a_lo[pb + i] : a * s.a_up[pb + i];
      beta = fmaf(fminf(a, 0.f), s.b_up[pb + i], beta);
      beta = fmaf(ah, s.bias[(unsigned)i / hw], beta);
      s.out[idx] = ah;
    }
  }
  red[w][lane] = beta;
  __syncthreads();
  if (w == 0 && ok) s.beta[q] = sgn * t.b[j] + ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
}

// Everything a call derives from the network, x0 and eps alone, in one launch: the exact
// layer-1 bounds and z1 = W1 x0 + b1, the per-neuron bias vectors of ReLU layers 2..L-1 and the
// transposed weights of the fully connected layers whose intermediate pass starts from them.
// Thread e is dealt to the segments in that order; a layer-1 neuron takes 16 threads.
struct SetupJob {
  DLayer t1;
  const float* x0;
  float eps;
  float* l1;    // [n1] lower, then [n1] upper bounds of h^(1)
  float* z1;
  long n1;
  int nfill;
  long fill_n[kMaxLayers];
  int fill_hw[kMaxLayers];
  const float* fill_b[kMaxLayers];
  float* fill_out[kMaxLayers];
  int ntr;
  const float* tr_W[kMaxLayers];
  int tr_out[kMaxLayers], tr_in[kMaxLayers];
  float* tr_dst[kMaxLayers];
  // the property merged into the last layer (Sec. 2.1): wsp[s][j] = (C W_L)[s][j], then
  // wsp[S n_{L-1} + s] = (C b_L)[s]; null when not needed
  float* wsp;
  const float* C;
  DLayer tL;
  int S;
};

// Neuron j of h^(1): row +-e_j carried through T_1 is +-W_1[j] (no relaxation in front of
// layer 1), so its bounds are z1_j -+ eps ||W_1[j]||_1 with z1_j = W_1[j] x0 + b_1[j] (Eq. 8; the
// taps of a convolution that fall on the zero padding are no entries of the row).  The 16 lanes
// of a group take every 16th entry and the sums meet in a fixed shuffle tree.
__device__ __forceinline__ void layer1_neuron(const SetupJob& job, long j, int g) {
  const DLayer& t = job.t1;
  float lin = 0.f, l1 = 0.f;
  if (t.kind == LIRPA_LINEAR) {
    for (int i = g; i < t.in_c; i += 16) {
      const float w = t.W[j * t.in_c + i];
      lin = fmaf(w, job.x0[i], lin);
      l1 += fabsf(w);
    }
  } else {
    const int hw = t.out_h * t.out_w, kk = t.k * t.k;
    const int co = (int)(j / hw), yo = (int)((j / t.out_w) % t.out_h), xo = (int)(j % t.out_w);
    for (int e = g; e < t.in_c * kk; e += 16) {
      const int ci = e / kk, ky = (e / t.k) % t.k, kx = e % t.k;
      const int yi = yo * t.stride - t.pad + ky, xi = xo * t.stride - t.pad + kx;
      if (yi < 0 || yi >= t.in_h || xi < 0 || xi >= t.in_w) continue;
      const float w = t.W[(long)co * t.in_c * kk + e];
      lin = fmaf(w, job.x0[((long)ci * t.in_h + yi) * t.in_w + xi], lin);
      l1 += fabsf(w);
    }
  }
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) {
    lin += __shfl_xor(lin, o, 64);
    l1 += __shfl_xor(l1, o, 64);
  }
  if (g == 0) {
    const float z = lin + t.b[j / (t.out_h * t.out_w)];
    job.z1[j] = z;
    job.l1[j] = z - job.eps * l1;
    job.l1[job.n1 + j] = z + job.eps * l1;
  }
}

__global__ void __launch_bounds__(kBlock) k_setup(SetupJob job) {
  long e = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (e < 16 * job.n1) {  // a group of 16 lanes never straddles the segment's end
    layer1_neuron(job, e >> 4, (int)(e & 15));
    return;
  }
  e -= 16 * job.n1;
  for (int f = 0; f < job.nfill; ++f) {
    if (e < job.fill_n[f]) {
      job.fill_out[f][e] = job.fill_b[f][e / job.fill_hw[f]];
      return;
    }
    e -= job.fill_n[f];
  }
  for (int k = 0; k < job.ntr; ++k) {
    const long nel = (long)job.tr_out[k] * job.tr_in[k];
    if (e < nel) {
      const long o = e / job.tr_in[k], i = e % job.tr_in[k];
      job.tr_dst[k][i * job.tr_out[k] + o] = job.tr_W[k][e];
      return;
    }
    e -= nel;
  }
  if (job.wsp) {
    const int nL = job.tL.out_c, nj = job.tL.in_c;
    if (e < (long)job.S * nj) {
      const int sr = (int)(e / nj), j = (int)(e % nj);
      float a = 0.f;
      for (int o = 0; o < nL; ++o) a = fmaf(job.C[sr * nL + o], job.tL.W[(long)o * nj + j], a);
      job.wsp[e] = a;
      return;
    }
    e -= (long)job.S * nj;
    if (e < job.S) {
      float a = 0.f;
      for (int o = 0; o < nL; ++o) a = fmaf(job.C[e * nL + o], job.tL.b[o], a);
      job.wsp[(long)job.S * nj + e] = a;
    }
  }
}

// Spec rows C_s over h^(L) (the property merged into the last layer): written to the slab as
// they are, with the bias C_s . b_L.
__global__ void __launch_bounds__(kBlock) k_spec_rows(const float* __restrict__ C, long nL,
                                                      const float* __restrict__ bL, int hwL,
                                                      long Q, long S, float* __restrict__ out,
                                                      long ldq, float* __restrict__ beta) {
  long q = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (q >= Q) return;
  long s = q % S;
  float acc = 0.f;
  for (long o = 0; o < nL; ++o) {
    float c = C[s * nL + o];
    out[o * ldq + q] = c;
    acc = fmaf(c, bL[o / hwL], acc);
  }
  beta[q] = acc;
}

// One backward step through a fully connected layer: a_in[i] = sum_o a_out[o] W[o][i].
template <int MODE>
__global__ void __launch_bounds__(kBlock) k_fcT(DLayer t, const float* __restrict__ in, long ldq,
                                                long Q, Sink s) {
  long q = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (q >= Q) return;
  long b = q / s.R, r = q % s.R;
  Acc acc{0.f, 0.f, 0.f};
  for (int i = 0; i < t.in_c; ++i) {
    float a = 0.f;
    for (int o = 0; o < t.out_c; ++o) a = fmaf(t.W[(long)o * t.in_c + i], in[o * ldq + q], a);
    sink_put<MODE>(s, acc, i, a, q, b);
  }
  sink_finish<MODE>(s, acc, q, b, r, false);
}

// One backward step through a convolution: the transposed convolution with the layer's own
// weights, stride and padding, gathered per input position.
template <int MODE>
__global__ void __launch_bounds__(kBlock) k_convT(DLayer t, const float* __restrict__ in,
                                                  long ldq, long Q, Sink s) {
  long q = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (q >= Q) return;
  long b = q / s.R, r = q % s.R;
  Acc acc{0.f, 0.f, 0.f};
  const int K = t.k, St = t.stride, P = t.pad;
  const long ohw = (long)t.out_h * t.out_w;
  const long wco = (long)t.in_c * K * K;
  for (int ci = 0; ci < t.in_c; ++ci)
    for (int yi = 0; yi < t.in_h; ++yi)
      for (int xi = 0; xi < t.in_w; ++xi) {
        float a = 0.f;
        for (int ky = 0; ky < K; ++ky) {
          int yn = yi + P - ky;
          if (yn < 0 || yn % St) continue;
          int yo = yn / St;
          if (yo >= t.out_h) continue;
          for (int kx = 0; kx < K; ++kx) {
            int xn = xi + P - kx;
            if (xn < 0 || xn % St) continue;
            int xo = xn / St;
            if (xo >= t.out_w) continue;
            const float* wp = t.W + ((long)ci * K + ky) * K + kx;
            const float* ip = in + ((long)yo * t.out_w + xo) * ldq + q;
            for (int co = 0; co < t.out_c; ++co) a = fmaf(wp[co * wco], ip[co * ohw * ldq], a);
          }
        }
        sink_put<MODE>(s, acc, ((long)ci * t.in_h + yi) * t.in_w + xi, a, q, b);
      }
  sink_finish<MODE>(s, acc, q, b, r, false);
}

// ---------------------------------------------------------------------------------------------
// MFMA stage kernels (fp32 32x32x2 matrix cores).
//
// Lane layout of v_mfma_f32_32x32x2_f32 (measured on gfx950): lane l supplies A[l%32][l/32] and
// B[l/32][l%32]; accumulator register r of lane l holds D[8(r/4) + 4(l/32) + r%4][l%32].
// ---------------------------------------------------------------------------------------------
typedef float floatx16 __attribute__((ext_vector_type(16)));

// Reduce (beta, lin, l1) of the two lane halves and of the waves of the block, then finish the
// rows q0..q0+31.  red: LDS scratch of nw*3*32 floats.
template <int MODE>
__device__ __forceinline__ void block_finish(const Sink& s, Acc acc, float* red, long q0, long Q,
                                             bool add_beta_from_acc) {
  const int lane = threadIdx.x & 63, wave = wave_id(), nw = blockDim.x >> 6;
  acc.beta += __shfl_xor(acc.beta, 32, 64);
  acc.lin += __shfl_xor(acc.lin, 32, 64);
  acc.l1 += __shfl_xor(acc.l1, 32, 64);
  if (lane < 32) {
    red[(wave * 3 + 0) * 32 + lane] = acc.beta;
    red[(wave * 3 + 1) * 32 + lane] = acc.lin;
    red[(wave * 3 + 2) * 32 + lane] = acc.l1;
  }
  __syncthreads();
  if (wave != 0 || lane >= 32) return;
  long q = q0 + lane;
  if (q >= Q) return;
  Acc t{0.f, 0.f, 0.f};
  for (int w = 0; w < nw; ++w) {
    t.beta += red[(w * 3 + 0) * 32 + lane];
    t.lin += red[(w * 3 + 1) * 32 + lane];
    t.l1 += red[(w * 3 + 2) * 32 + lane];
  }
  (void)add_beta_from_acc;
  sink_finish<MODE>(s, t, q, q / s.R, q % s.R, false);
}

// Transposed convolution as a scatter-form implicit GEMM on 16x16x4 MFMA.
//
// Lane layout of v_mfma_f32_16x16x4_f32 (measured on gfx950): lane l supplies A[l%16][l/16] and
// B[l/16][l%16]; accumulator register r of lane l holds D[4(l/16) + r][l%16].
//
// Block: 16 rows q (N) and one wave per CPW output channels ci.  M = 16 tap slots (G, kx): lane
// group G = l/16, kx = register r; K = 4 of the layer's output channels co per MFMA.  Input
// positions are visited row by row (y1) from a double-buffered LDS tile.  Output row y always
// lives in lane group (y + P) mod K, so at input row y1 group G takes tap row
// ky = (G - y1*S) mod K (the A operand rotates, the accumulators stay put) and collects in its
// own registers the whole contribution of row y1 to output row y1*S - P + ky, including the
// overlap along x.  Rows with ky < S are complete after row y1 and go to the epilogue
// (relaxation of layer m-1 plus bias, or concretisation) before the group starts its next row.
// The y1 loop is unrolled over the rotation period so every register index is static.
template <int K, int S, int P, int H1, int W1, int H0, int W0, int CO, int CPW, int NW,
          int MODE, bool TAPE>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(MODE == MODE_BOUND && !TAPE ? (CO <= 8 ? 4 : 3) : 1, MODE == MODE_BOUND && !TAPE ? 8 : 2)))
k_convT_mfma(DLayer t, const float* __restrict__ in, unsigned ldq, unsigned Q, Sink s) {
  static_assert(K <= 4 && S <= K && CO % 4 == 0 && W0 % 4 == 0, "unsupported geometry");
  constexpr int KS = CO / 4;
  constexpr int NT = 64 * NW;
  constexpr int PER = (K % S == 0) ? K / S : K;  // rotation period of the tap rows
  // LDS tile of one input row, [CO][W1][16] with each channel padded to a stride of 16 mod 64
  // floats, so the four lane groups of a B-operand read (channels 4ks + G) hit disjoint banks
  constexpr int CS = W1 * 16 + (80 - (W1 * 16) % 64) % 64;
  constexpr int TILE = CO * CS;       // floats per input-row tile
  constexpr int NV4 = CO * W1 * 4;    // float4 per tile
  extern __shared__ float lds[];
  float* tiles = lds;                  // 2 x [CO][W1][16]
  float* xs = lds + 2 * TILE;          // MODE_BOUND: x0 [in_c*H0*W0]
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int n = lane & 15, G = lane >> 4;
  const unsigned q0 = xcd_tile(blockIdx.x) * 16u;
  if (q0 >= Q) return;  // grid padding, uniform per block
  const unsigned q = q0 + n;
  const bool qok = q < Q;
  const unsigned b = qok ? q / (unsigned)s.R : 0u;
  float* red = xs + (MODE == MODE_BOUND && s.x0 ? t.in_c * H0 * W0 : 0);  // [NW][3][16]

  const bool with_x0 = MODE == MODE_BOUND && s.x0 != nullptr;
  if (with_x0) {
    const int nx = t.in_c * H0 * W0;
    for (int e = threadIdx.x; e < nx; e += NT) xs[e] = s.x0[e];
  }

  // A operands, one set per rotation phase: slot (M/4, M%4) of lane l (M = l%16) takes tap
  // ((M/4 - ph*S) mod K, M%4) of co = 4*ks + l/16
  float wreg[PER][CPW][KS];
  int cis[CPW];
  bool cok[CPW];
#pragma unroll
  for (int c = 0; c < CPW; ++c) {
    cis[c] = wave * CPW + c;
    cok[c] = cis[c] < t.in_c;
  }
  {
    const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
    for (int ph = 0; ph < PER; ++ph) {
      const int ky = ((slot - ph * S) % K + K) % K;
#pragma unroll
      for (int c = 0; c < CPW; ++c)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int co = 4 * ks + G;
          wreg[ph][c][ks] = (cok[c] && slot < K && kx < K)
                                ? t.W[((co * t.in_c + cis[c]) * K + ky) * K + kx] : 0.f;
        }
    }
  }

  float beta = 0.f, lin = 0.f, l1 = 0.f;
  // Relaxation parameters of one output row (MODE_SLAB): loaded before the MFMAs of the step
  // that completes the row, so their latency hides behind the matrix work.
  constexpr int NQ = W0 / 4;
  constexpr int NP = MODE == MODE_SLAB ? NQ : 1;
  // early loads only where the registers allow it; otherwise just before the row is relaxed
  constexpr bool EARLY = MODE == MODE_SLAB && CPW == 1 && W0 <= 16;
  float4v p_lo[CPW][NP], p_up[CPW][NP], p_bu[CPW][NP], p_bz[CPW][NP];
  auto load_row = [&](int c, int y) {
    if constexpr (EARLY) {
      if (!cok[c] || !qok || y < 0 || y >= H0) return;
      const unsigned rowi = ((unsigned)cis[c] * H0 + y) * W0;
      const long pb = (long)b * s.pstride + rowi;
#pragma unroll
      for (int i = 0; i < NQ; ++i) {
        p_lo[c][i] = *reinterpret_cast<const float4v*>(s.a_lo + pb + 4 * i);
        p_up[c][i] = *reinterpret_cast<const float4v*>(s.a_up + pb + 4 * i);
        p_bu[c][i] = *reinterpret_cast<const float4v*>(s.b_up + pb + 4 * i);
        p_bz[c][i] = *reinterpret_cast<const float4v*>(s.bias + rowi + 4 * i);
      }
    }
  };
  auto emit = [&](int c, int y, const float* vals) {
    if (!cok[c] || !qok || y < 0 || y >= H0) return;
    const unsigned rowi = ((unsigned)cis[c] * H0 + y) * W0;
    if constexpr (MODE == MODE_BOUND) {
      if (with_x0) {
#pragma unroll
        for (int x = 0; x < W0; ++x) {
          const float a = vals[x];
          if constexpr (TAPE) s.tsign[(rowi + x) * ldq + q] = sign8(a);
          lin = fmaf(a, xs[rowi + x], lin);
          l1 += fabsf(a);
        }
      } else {
#pragma unroll
        for (int x = 0; x < W0; ++x) {
          if constexpr (TAPE) s.tsign[(rowi + x) * ldq + q] = sign8(vals[x]);
          l1 += fabsf(vals[x]);
        }
      }
    } else {
      const long pb = (long)b * s.pstride + rowi;
#pragma unroll
      for (int i = 0; i < NQ; ++i) {
        float4v lo, up, bu, bz;
        if constexpr (EARLY) {
          lo = p_lo[c][i];
          up = p_up[c][i];
          bu = p_bu[c][i];
          bz = p_bz[c][i];
        } else {
          lo = *reinterpret_cast<const float4v*>(s.a_lo + pb + 4 * i);
          up = *reinterpret_cast<const float4v*>(s.a_up + pb + 4 * i);
          bu = *reinterpret_cast<const float4v*>(s.b_up + pb + 4 * i);
          bz = *reinterpret_cast<const float4v*>(s.bias + rowi + 4 * i);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float a = vals[4 * i + j];
          const unsigned idx = (rowi + 4 * i + j) * ldq + q;
          if constexpr (TAPE) s.tape[idx] = a;
          const float ah = a >= 0.f ? a * lo[j] : a * up[j];
          beta = fmaf(fminf(a, 0.f), bu[j], beta);
          beta = fmaf(ah, bz[j], beta);
          s.out[idx] = ah;
        }
      }
    }
  };

  float acc[CPW][W0];
#pragma unroll
  for (int c = 0; c < CPW; ++c)
#pragma unroll
    for (int x = 0; x < W0; ++x) acc[c][x] = 0.f;
  // Stride 2 (bound stages): the four output columns x1*2 - P + kx of input column x1 do not
  // overlap those of x1 + 2, so the MFMAs accumulate in place -- one float4 per input column
  // x1, in two interleaved families (x1 even, x1 odd) -- and a row is summed from the two
  // families only when it is complete, instead of after every MFMA.
  constexpr bool DIRECT = MODE == MODE_BOUND && S == 2;
  constexpr int NB = (W1 + 1) / 2;
  float4v accd[DIRECT ? CPW : 1][2][DIRECT ? NB : 1];
  if constexpr (DIRECT) {
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int m = 0; m < NB; ++m) accd[c][f][m] = float4v{0.f, 0.f, 0.f, 0.f};
  }
  // row of channel c from the two families (column x: x1 = 2m + f with 4m + kx = x + P - 2f)
  auto gather = [&](int c, float* vals) {
    if constexpr (DIRECT) {
#pragma unroll
      for (int x = 0; x < W0; ++x) {
        float v = 0.f;
#pragma unroll
        for (int f = 0; f < 2; ++f) {
          const int tt = x + P - 2 * f;
          if (tt >= 0 && (tt >> 2) < NB && 2 * (tt >> 2) + f < W1) v += accd[c][f][tt >> 2][tt & 3];
        }
        vals[x] = v;
      }
    }
  };
  auto reset = [&](int c) {
    if constexpr (DIRECT) {
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int m = 0; m < NB; ++m) accd[c][f][m] = float4v{0.f, 0.f, 0.f, 0.f};
    } else {
#pragma unroll
      for (int x = 0; x < W0; ++x) acc[c][x] = 0.f;
    }
  };

  auto gaddr = [&](int y1, int v4) {
    const int cx = v4 >> 2, j4 = v4 & 3;
    const int co = cx / W1, x1 = cx - co * W1;
    return in + ((unsigned)(co * H1 + y1) * W1 + x1) * ldq + q0 + j4 * 4;
  };
  auto loff = [&](int v4) {
    const int cx = v4 >> 2, j4 = v4 & 3;
    const int co = cx / W1, x1 = cx - co * W1;
    return co * CS + x1 * 16 + j4 * 4;
  };
  for (int v4 = threadIdx.x; v4 < NV4; v4 += NT)
    *reinterpret_cast<float4v*>(tiles + loff(v4)) = *reinterpret_cast<const float4v*>(gaddr(0, v4));
  __syncthreads();

  // Per input row: (1) issue the loads of the next input tile and of the parameters of the
  // rows this step completes, (2) the MFMAs, (3) park the next tile in LDS, (4) relax and store
  // the completed rows, (5) an LDS-only barrier.  No wait inside the loop covers the global
  // stores of (4).
  constexpr int PF = (NV4 + NT - 1) / NT;  // prefetched float4 per thread
  for (int ybase = 0; ybase < H1; ybase += PER) {
#pragma unroll
    for (int ph = 0; ph < PER; ++ph) {
      const int y1 = ybase + ph;
      if (H1 % PER != 0 && y1 >= H1) break;
      const float* tile = tiles + (y1 & 1) * TILE;
      const bool more = y1 + 1 < H1;
      // this lane group's tap row at this phase; rows with ky < S are complete after it
      const int ky = ((G - ph * S) % K + K) % K;
      const bool done = G < K && ky < S;
      const int yout = y1 * S - P + ky;
      float4v pf[PF];
      {
        const int yn = more ? y1 + 1 : y1;
#pragma unroll
        for (int k = 0; k < PF; ++k) {
          const int v4 = min((int)threadIdx.x + k * NT, NV4 - 1);
          pf[k] = *reinterpret_cast<const float4v*>(gaddr(yn, v4));
        }
      }
      if (EARLY && done) {
#pragma unroll
        for (int c = 0; c < CPW; ++c) load_row(c, yout);
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the loads above ahead of the matrix work
#pragma unroll
      for (int x1 = 0; x1 < W1; ++x1) {
        float bv[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) bv[ks] = tile[(4 * ks + G) * CS + x1 * 16 + n];
#pragma unroll
        for (int c = 0; c < CPW; ++c) {
          if constexpr (DIRECT) {
            float4v d = accd[c][x1 & 1][x1 >> 1];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ph][c][ks], bv[ks], d, 0, 0, 0);
            accd[c][x1 & 1][x1 >> 1] = d;
          } else {
            float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ph][c][ks], bv[ks], d, 0, 0, 0);
#pragma unroll
            for (int kx = 0; kx < K; ++kx) {
              const int col = x1 * S - P + kx;
              if (col >= 0 && col < W0) acc[c][col] += d[kx];
            }
          }
        }
      }
      if (more) {
        float* nt = tiles + ((y1 + 1) & 1) * TILE;
#pragma unroll
        for (int k = 0; k < PF; ++k) {
          const int v4 = (int)threadIdx.x + k * NT;
          if (v4 < NV4) *reinterpret_cast<float4v*>(nt + loff(v4)) = pf[k];
        }
      }
      if (done) {
#pragma unroll
        for (int c = 0; c < CPW; ++c) {
          if constexpr (DIRECT) {
            float vals[W0];
            gather(c, vals);
            emit(c, yout, vals);
          } else {
            emit(c, yout, acc[c]);
          }
          reset(c);
        }
      }
      if (more) lds_barrier();
    }
  }
  {
    // rows still open after the last input row are complete too
    constexpr int ph_last = (H1 - 1) % PER;
    const int ky = ((G - ph_last * S) % K + K) % K;
    if (G < K && ky >= S) {
#pragma unroll
      for (int c = 0; c < CPW; ++c) {
        load_row(c, (H1 - 1) * S - P + ky);
        if constexpr (DIRECT) {
          float vals[W0];
          gather(c, vals);
          emit(c, (H1 - 1) * S - P + ky, vals);
        } else {
          emit(c, (H1 - 1) * S - P + ky, acc[c]);
        }
      }
    }
  }
  // output rows no input row reaches (zero coefficients)
  constexpr int YZ = (H1 - 1) * S - P + K;
  if constexpr (YZ < H0) {
    if (G == 0) {
      float zero[W0];
#pragma unroll
      for (int x = 0; x < W0; ++x) zero[x] = 0.f;
#pragma unroll
      for (int y = YZ; y < H0; ++y)
#pragma unroll
        for (int c = 0; c < CPW; ++c) {
          load_row(c, y);
          emit(c, y, zero);
        }
    }
  }

  // sum over lane groups and waves, then finish rows q0..q0+15
  beta += __shfl_xor(beta, 16, 64);
  lin += __shfl_xor(lin, 16, 64);
  l1 += __shfl_xor(l1, 16, 64);
  beta += __shfl_xor(beta, 32, 64);
  lin += __shfl_xor(lin, 32, 64);
  l1 += __shfl_xor(l1, 32, 64);
  __syncthreads();
  if (lane < 16) {
    red[(wave * 3 + 0) * 16 + lane] = beta;
    red[(wave * 3 + 1) * 16 + lane] = lin;
    red[(wave * 3 + 2) * 16 + lane] = l1;
  }
  __syncthreads();
  if (wave != 0 || lane >= 16 || !qok) return;
  Acc tot{0.f, 0.f, 0.f};
  for (int w = 0; w < NW; ++w) {
    tot.beta += red[(w * 3 + 0) * 16 + lane];
    tot.lin += red[(w * 3 + 1) * 16 + lane];
    tot.l1 += red[(w * 3 + 2) * 16 + lane];
  }
  sink_finish<MODE>(s, tot, q, b, q % (unsigned)s.R, false);
}

// Transposed convolution with the relaxation of layer m-1 fused, on specialised waves.
//
// The rotating lane-group MFMA scheme of k_convT_mfma, with the epilogue moved off the matrix
// waves.  NM = CI / CPW "matrix" waves own CPW output channels each: per input row they read the
// B operands from the LDS tile, run the MFMAs, and park the output rows that row completes,
// unrelaxed, in an LDS row buffer.  They also issue every global load of the block -- the next
// input tile and the relaxation parameters of the rows they complete (staged into LDS one step
// ahead) -- and no global store.  NS "storer" waves take the parked rows of the previous step:
// relaxation (Eq. 6), intercept and bias terms of each row, and the stores of the relaxed
// coefficients; they issue no global load.  So no wave ever waits on a counter that also covers
// global stores, and the matrix waves never wait on the relaxation's arithmetic.  One LDS-only
// barrier per input row hands the buffers over (double-buffered).  A block takes 16 rows q
// spanning at most two sub-domains (R >= 16).
// FC: the stage opens a pass at the fully connected layer above (see FcSrc).  The matrix waves
// then build each input tile themselves, one step ahead: the rows of W_k and the relaxation of
// this stage's own layer are loaded into registers before the MFMAs of the current row and
// turned into relaxed coefficients (with their intercept and bias terms) after them.  The slab
// that would hold these coefficients is never written or read.
template <int K, int S, int P, int H1, int W1, int H0, int W0, int CO, int CI, int CPW, int NS,
          bool TAPE, bool FC>
__global__ void __launch_bounds__(64 * (CI / CPW + NS), CI / CPW + NS <= 8 ? 4 : (CI / CPW + NS <= 12 ? 6 : 1))
    k_convT_relax_ws(DLayer t, const float* __restrict__ in, unsigned ldq, unsigned Q, Sink s,
                     FcSrc fc) {
  static_assert(W0 == 16 && K <= 4 && S <= K && CO % 4 == 0 && CI % CPW == 0, "geometry");
  static_assert((H1 - 1) * S - P + K >= H0, "every output row is reached by an input row");
  constexpr int NM = CI / CPW;                   // matrix waves
  constexpr int NTM = 64 * NM;
  constexpr int KS = CO / 4;
  constexpr int PER = (K % S == 0) ? K / S : K;  // rotation period of the tap rows
  // tile: [W1][CO][16 q], so that the four lane groups of a B-operand read (channels 4ks + G
  // at one x1) cover 64 consecutive floats
  constexpr int TILE = W1 * CO * 16;
  constexpr int NV4 = CO * W1 * 4;               // float4 per input tile
  constexpr int PF = (NV4 + NTM - 1) / NTM;
  constexpr int RSL = S > K - S ? S : K - S;     // output rows completed per step (max)
  constexpr int RB = RSL * CI * 16 * 16;         // row buffer: [RSL][CI][16 q][16 x]
  constexpr int AST = RSL * CI * W0;             // one parameter array of a stage
  constexpr int PB = 7 * AST;                    // [a_lo, a_up, b_up] x 2 sub-domains + bias
  constexpr int NPV4 = PB / 4;
  constexpr int PP = (NPV4 + NTM - 1) / NTM;
  static_assert(AST % 256 == 0 && NV4 % 64 == 0, "DMA chunks must be whole waves");
  static_assert(!FC || W1 % 4 == 0, "FC source: float4 quads of x1");
  // FC source: task tk of an input row = (quad qd of four consecutive x1 of channel co, pair of
  // rows q0 + 2 qp, q0 + 2 qp + 1), qd = t4 * CO + co, tk = 8 qd + qp
  constexpr int NTASK = CO * W1 / 4 * 8;
  constexpr int TPL = FC ? (NTASK + NTM - 1) / NTM : 1;
  // Input tiles and relaxation parameters reach LDS by DMA (global_load_lds), issued by the
  // matrix waves two steps ahead of their use and waited for, per wave, just before the
  // barrier that publishes them.  They are issued from inline assembly, so the compiler neither
  // holds registers for them nor orders other LDS accesses behind them.
  __shared__ float tiles[3][TILE];
  __shared__ float rows[2][RB];
  __shared__ float pars[3][PB];
  __shared__ float red[NS * 16];
  __shared__ float red_fc[FC ? NM * 16 : 1];

  const int lane = threadIdx.x & 63, wave = wave_id();
  const unsigned q0 = xcd_tile(blockIdx.x) * 16u;
  if (q0 >= Q) return;  // grid padding, uniform per block
  const unsigned R = (unsigned)s.R;
  const unsigned b0 = q0 / R;
  const unsigned b1 = (min(q0 + 15u, Q - 1u)) / R;  // b0 or b0 + 1

  // output row of slot r at stage e (stage H1: the rows still open after the last input row)
  auto yrow = [&](int e, int r) { return e < H1 ? e * S - P + r : (H1 - 1) * S - P + S + r; };
  auto nrows = [&](int e) { return e < H1 ? S : K - S; };

  if (wave < NM) {
    // ------------------------------------------------------------------ matrix waves
    const int n = lane & 15, G = lane >> 4;
    const int tid = threadIdx.x;  // < NTM
    float wreg[PER][CPW][KS];
    {
      const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
      for (int ph = 0; ph < PER; ++ph) {
        const int ky = ((slot - ph * S) % K + K) % K;
#pragma unroll
        for (int c = 0; c < CPW; ++c)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const int co = 4 * ks + G, ci = wave * CPW + c;
            wreg[ph][c][ks] = (slot < K && kx < K)
                                  ? t.W[((co * CI + ci) * K + ky) * K + kx] : 0.f;
          }
      }
    }
    // 16 bytes per lane from src into LDS at base + 16 * lane (base uniform over the wave)
    auto dma16 = [&](const float* src, const float* base) {
      const unsigned lds = __builtin_amdgcn_readfirstlane(
          (unsigned)(size_t)(__attribute__((address_space(3))) const float*)base);
      asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                   :: "v"(src), "s"(lds) : "memory", "m0");
    };
    auto dma_tile = [&](float* buf, int y1) {  // input row y1 into buf
#pragma unroll
      for (int k = 0; k < PF; ++k) {
        const int v4 = tid + k * NTM;  // whole waves in or out of range
        if (v4 < NV4) {
          const int cx = v4 >> 2, j4 = v4 & 3;
          const int x1 = cx / CO, co = cx - x1 * CO;
          dma16(in + ((unsigned)(co * H1 + y1) * W1 + x1) * ldq + q0 + j4 * 4,
                buf + 4 * (v4 - lane));
        }
      }
    };
    // parameters of stage e into pbuf: float4 v of [arr][RSL][CI][W0/4], arr = 3 bsel + {0,1,2}
    // for a_lo, a_up, b_up of sub-domain b0 + bsel, arr = 6 for the bias.  Entries of rows
    // outside the map or of a second sub-domain the block does not have are never read: they
    // fetch the bias instead.
    auto dma_pars = [&](float* pbuf, int e) {
#pragma unroll
      for (int k = 0; k < PP; ++k) {
        const int v = tid + k * NTM;
        if (v < NPV4) {
          const int x4 = v % (W0 / 4);
          const int c = (v / (W0 / 4)) % CI;
          const int r = (v / (W0 / 4 * CI)) % RSL;
          const int arr = __builtin_amdgcn_readfirstlane(v >> 6) / (AST / 256);
          const int bsel = arr < 6 ? arr / 3 : 0;
          const int y = yrow(e, r);
          const bool ok = r < nrows(e) && y >= 0 && y < H0 && b0 + bsel <= b1;
          const unsigned rowi = ok ? ((unsigned)c * H0 + y) * W0 + 4 * x4 : 0u;
          const long pb = (long)(b0 + bsel) * s.pstride + rowi;
          const float* src = s.bias + rowi;
          if (ok && arr < 6) {
            switch (arr % 3) {
              case 0: src = s.a_lo + pb; break;
              case 1: src = s.a_up + pb; break;
              default: src = s.b_up + pb; break;
            }
          }
          dma16(src, pbuf + 4 * (v - lane));
        }
      }
    };
    // DMA instructions this wave issues per call of dma_pars and dma_tile (whole waves)
    int npw = 0, ntw = 0;
#pragma unroll
    for (int k = 0; k < PP; ++k) npw += (wave * 64 + k * NTM < NPV4) ? 1 : 0;
#pragma unroll
    for (int k = 0; k < PF; ++k) ntw += (wave * 64 + k * NTM < NV4) ? 1 : 0;
    // wait until at most n of this wave's DMAs are outstanding (n is uniform, <= PP + PF)
    auto wait_dma = [](int n) {
      switch (n) {
        case 0: __builtin_amdgcn_s_waitcnt(0xF70); break;
        case 1: __builtin_amdgcn_s_waitcnt(0xF71); break;
        case 2: __builtin_amdgcn_s_waitcnt(0xF72); break;
        case 3: __builtin_amdgcn_s_waitcnt(0xF73); break;
        default: __builtin_amdgcn_s_waitcnt(0xF74); break;
      }
    };
    static_assert(PP + PF <= 4, "wait_dma covers at most four DMAs in flight");
    // a parked row of 16 x values holds its float4 i at position i ^ (q >> 2), so that the 16
    // rows q of one write (64 bytes apart) spread over all banks
    auto park = [&](int slot, int r, int c, const float* v) {
      float* dst = rows[slot] + (((r * CI + wave * CPW + c) * 16 + n) * 16);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<float4v*>(dst + 4 * (i ^ (n >> 2))) =
            float4v{v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]};
    };

    // FC source: per task, the fixed part of its addresses and its sign (0 for rows past Q)
    typedef float float2v __attribute__((ext_vector_type(2)));
    unsigned g_wa[TPL], g_wb[TPL], g_pb[TPL];  // offsets into W_k and the parameter arrays
    float g_sa[TPL], g_sb[TPL], g_bz[TPL];
    int g_lds[TPL];
    bool g_on[TPL];
    float4v g_xa[TPL], g_xb[TPL], g_lo[TPL], g_up[TPL], g_bu[TPL];
    float fbeta_a = 0.f, fbeta_b = 0.f;
    if constexpr (FC) {
      const unsigned nin = CO * H1 * W1, nk = (unsigned)fc.nk;
#pragma unroll
      for (int k = 0; k < TPL; ++k) {
        const int tk = tid + k * NTM;
        g_on[k] = tk < NTASK;
        const int qp = tk & 7, qd = g_on[k] ? tk >> 3 : 0;
        const int co = qd % CO, t4 = qd / CO;
        const unsigned qa = q0 + 2u * qp, qb = qa + 1u;
        const unsigned ra = qa % R, rb = qb % R;
        g_sa[k] = qa < Q ? (ra < nk ? 1.f : -1.f) : 0.f;
        g_sb[k] = qb < Q ? (rb < nk ? 1.f : -1.f) : 0.f;
        const unsigned i0 = (unsigned)co * H1 * W1 + 4u * t4;
        g_wa[k] = (ra % nk) * nin + i0;
        g_wb[k] = (rb % nk) * nin + i0;
        // R is even, so rows 2 qp and 2 qp + 1 share their sub-domain
        g_pb[k] = (qa < Q ? qa / R : b0) * (unsigned)s.pstride + i0;
        g_bz[k] = t.b[co];
        g_lds[k] = (4 * t4 * CO + co) * 16 + 2 * qp;
      }
    }
    auto gen_load = [&](int yg) {
#pragma unroll
      for (int k = 0; k < TPL; ++k)
        if (g_on[k]) {
          const unsigned o = (unsigned)yg * W1;
          g_xa[k] = *reinterpret_cast<const float4v*>(fc.W + (g_wa[k] + o));
          g_xb[k] = *reinterpret_cast<const float4v*>(fc.W + (g_wb[k] + o));
          g_lo[k] = *reinterpret_cast<const float4v*>(fc.a_lo + (g_pb[k] + o));
          g_up[k] = *reinterpret_cast<const float4v*>(fc.a_up + (g_pb[k] + o));
          g_bu[k] = *reinterpret_cast<const float4v*>(fc.b_up + (g_pb[k] + o));
        }
    };
    // relaxation (Eq. 6) of the loaded coefficients into tile buf, with the intercept and bias
    // terms of rows 2 qp and 2 qp + 1
    auto gen_store = [&](float* buf) {
#pragma unroll
      for (int k = 0; k < TPL; ++k)
        if (g_on[k]) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float a = g_sa[k] * g_xa[k][e], b = g_sb[k] * g_xb[k][e];
            const float ha = a * (a >= 0.f ? g_lo[k][e] : g_up[k][e]);
            const float hb = b * (b >= 0.f ? g_lo[k][e] : g_up[k][e]);
            fbeta_a = fmaf(fminf(a, 0.f), g_bu[k][e], fbeta_a);
            fbeta_a = fmaf(ha, g_bz[k], fbeta_a);
            fbeta_b = fmaf(fminf(b, 0.f), g_bu[k][e], fbeta_b);
            fbeta_b = fmaf(hb, g_bz[k], fbeta_b);
            *reinterpret_cast<float2v*>(buf + g_lds[k] + e * CO * 16) = float2v{ha, hb};
          }
        }
    };

    // prologue: parameters of stage 0, input rows 0 and 1; row 0 and the parameters landed
    dma_pars(pars[0], 0);
    if constexpr (FC) {
      gen_load(0);
      gen_store(tiles[0]);
      wait_dma(0);
    } else {
      dma_tile(tiles[0], 0);
      if (H1 > 1) {
        dma_tile(tiles[1], 1);
        wait_dma(ntw);
      } else {
        wait_dma(0);
      }
    }
    lds_barrier();

    float acc[CPW][W0];
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int x = 0; x < W0; ++x) acc[c][x] = 0.f;

    // Step y1: DMA the parameters of stage y1+1 and input row y1+2; MFMAs on row y1; park the
    // rows it completes; wait for this wave's DMAs of earlier steps (row y1+1, parameters of
    // stage y1); barrier.  Unrolled over U steps so that the buffer indices are constants.
    constexpr int U = PER % 3 == 0 ? PER : 3 * PER;
    for (int ybase = 0; ybase < H1; ybase += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int y1 = ybase + u;
        if (H1 % U != 0 && y1 >= H1) break;
        const int ph = u % PER;
        const float* tile = tiles[u % 3];
        dma_pars(pars[(u + 1) % 3], y1 + 1);
        const bool more = y1 + 2 < H1;
        if constexpr (FC) {
          if (y1 + 1 < H1) gen_load(y1 + 1);
        } else if (more) {
          dma_tile(tiles[(u + 2) % 3], y1 + 2);
        }
#pragma unroll
        for (int x1 = 0; x1 < W1; ++x1) {
          float bv[KS];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) bv[ks] = tile[(x1 * CO + 4 * ks + G) * 16 + n];
#pragma unroll
          for (int c = 0; c < CPW; ++c) {
            float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ph][c][ks], bv[ks], d, 0, 0, 0);
#pragma unroll
            for (int kx = 0; kx < K; ++kx) {
              const int col = x1 * S - P + kx;
              if (col >= 0 && col < W0) acc[c][col] += d[kx];
            }
          }
        }
        const int ky = ((G - ph * S) % K + K) % K;
        if (G < K && ky < S) {
#pragma unroll
          for (int c = 0; c < CPW; ++c) {
            park(y1 & 1, ky, c, acc[c]);
#pragma unroll
            for (int x = 0; x < W0; ++x) acc[c][x] = 0.f;
          }
        }
        if constexpr (FC) {
          if (y1 + 1 < H1) gen_store(tiles[(u + 1) % 3]);
          wait_dma(0);
        } else {
          wait_dma(npw + (more ? ntw : 0));
        }
        lds_barrier();
      }
    }
    // stage H1: the rows still open; its parameters were fetched at the last step
    wait_dma(0);
    {
      constexpr int ph_last = (H1 - 1) % PER;
      const int ky = ((G - ph_last * S) % K + K) % K;
      if (G < K && ky >= S) {
#pragma unroll
        for (int c = 0; c < CPW; ++c) park(H1 & 1, ky - S, c, acc[c]);
      }
    }
    lds_barrier();
    if constexpr (FC) {
      // rows 2 qp, 2 qp + 1 of every task of this wave: lanes qp, qp + 8, ..., qp + 56
#pragma unroll
      for (int o = 8; o < 64; o <<= 1) {
        fbeta_a += __shfl_xor(fbeta_a, o, 64);
        fbeta_b += __shfl_xor(fbeta_b, o, 64);
      }
      if (lane < 8) {
        red_fc[wave * 16 + 2 * lane] = fbeta_a;
        red_fc[wave * 16 + 2 * lane + 1] = fbeta_b;
      }
    }
    lds_barrier();  // the storers' final reduction
    return;
  }

  // -------------------------------------------------------------------- storer waves
  const int ws = wave - NM;
  const int qn = lane & 15, xg = lane >> 4;
  const unsigned q = q0 + qn;
  const bool qok = q < Q;
  const int bsel = qok ? (int)(q / R - b0) : 0;
  // Rows q0..q0+15 all lie inside the slab's padded width (ldq is a multiple of 64), so rows
  // past Q are stored too (never read as results) and the stores need no lane mask.  A store
  // address is a block-uniform row base plus this lane's 32-bit byte offset.
  const unsigned lane_boff = (4u * xg * ldq + qn) * 4u;
  float beta = 0.f;
  auto stage = [&](int e) {
    const int slot = e & 1;
    const float* pst = pars[e % 3];
    const int nr = nrows(e);
    for (int it = ws; it < nr * CI; it += NS) {
      const int r = it / CI, c = it - r * CI;
      const int y = yrow(e, r);
      if (y < 0 || y >= H0) continue;
      const float4v a = *reinterpret_cast<const float4v*>(
          rows[slot] + ((r * CI + c) * 16 + qn) * 16 + 4 * (xg ^ (qn >> 2)));
      const int off = r * CI * W0 + c * W0 + 4 * xg;
      const float4v lo = *reinterpret_cast<const float4v*>(pst + (3 * bsel + 0) * AST + off);
      const float4v up = *reinterpret_cast<const float4v*>(pst + (3 * bsel + 1) * AST + off);
      const float4v bu = *reinterpret_cast<const float4v*>(pst + (3 * bsel + 2) * AST + off);
      const float4v bz = *reinterpret_cast<const float4v*>(pst + 6 * AST + off);
      const unsigned row0 = ((unsigned)c * H0 + y) * W0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const size_t base = (size_t)(row0 + j) * ldq + q0;  // uniform
        if constexpr (TAPE) store_row(s.tape + base, lane_boff, a[j]);
        const bool pos = a[j] >= 0.f;
        const float ah = a[j] * (pos ? lo[j] : up[j]);
        beta = fmaf(pos ? 0.f : a[j], bu[j], beta);
        beta = fmaf(ah, bz[j], beta);
        store_row(s.out + base, lane_boff, ah);
      }
    }
  };
  lds_barrier();  // initial tile
  for (int y1 = 0; y1 < H1; ++y1) {
    if (y1 > 0) stage(y1 - 1);
    lds_barrier();
  }
  stage(H1 - 1);
  lds_barrier();
  stage(H1);
  beta += __shfl_xor(beta, 16, 64);
  beta += __shfl_xor(beta, 32, 64);
  if (lane < 16) red[ws * 16 + lane] = beta;
  lds_barrier();
  if (ws != 0 || lane >= 16 || !qok) return;
  float tot = 0.f;
  for (int w = 0; w < NS; ++w) tot += red[w * 16 + lane];
  if constexpr (FC) {
    // the rows' own bias +-b_k[j] and the terms of the relaxation that built them
    const unsigned r = q % R, nk = (unsigned)fc.nk;
    float fb = r < nk ? fc.b[r] : -fc.b[r - nk];
    for (int w = 0; w < NM; ++w) fb += red_fc[w * 16 + lane];
    tot += fb;
  }
  Acc a{tot, 0.f, 0.f};
  sink_finish<MODE_SLAB>(s, a, q, q / R, q % R, FC);
}

// The last two backward stages of a pass fused: T_2^T with the relaxation of layer 1, then T_1^T
// with the concretisation (Eq. 6-8), for 16 rows per block.  The coefficients over g^(1) never
// leave LDS.  Wave roles, all of them stepping through the same barriers t = 0 .. H1 + 2:
//   matrix waves (one per channel of g^(1)): T_2^T on input row t as in k_convT_relax_ws; the
//     rows over g^(1) completed at step t ("stage t"; stage H1 = the rows still open after the
//     last input row) are parked, unrelaxed, in slot t mod 3 of an LDS ring, and the layer-1
//     relaxation parameters of stage t are staged in LDS; every global load is theirs;
//   storer waves: relax stage t-1 in place (Eq. 6) and accumulate each row's intercept and bias
//     terms;
//   x waves (one per input channel of T_1): T_1^T over the rows of stage t-2, in increasing
//     order, with the rotating lane-group scheme, accumulating ||A_x||_1 per row.
// The bound of each row is then beta - eps ||A_x||_1 (the linear term sits in the layer-1 bias).
template <int K, int S, int P, int H1, int W1, int H0, int W0, int CO, int CI, int NS, int K1,
          int S1, int P1, int HX, int WX, int C0>
__global__ void __launch_bounds__(64 * (CI + NS + C0))
    k_convT2_bound(DLayer t, DLayer t1, const float* __restrict__ in, unsigned ldq, unsigned Q,
                   Sink s) {
  static_assert(W0 == 16 && K <= 4 && S <= K && CO % 4 == 0 && CI % 4 == 0, "geometry");
  static_assert(K1 <= 4 && S1 <= K1 && WX % 4 == 0, "geometry");
  static_assert((H1 - 1) * S - P + K >= H0, "every output row is reached by an input row");
  static_assert((H0 - 1) * S1 - P1 + K1 >= HX, "every input row of T_1 is reached");
  constexpr int NM = CI;                         // matrix waves
  constexpr int NTM = 64 * NM;
  constexpr int KS = CO / 4, KS1 = CI / 4;
  constexpr int PER = (K % S == 0) ? K / S : K;
  constexpr int PER1 = (K1 % S1 == 0) ? K1 / S1 : K1;
  constexpr int CS = W1 * 16 + (80 - (W1 * 16) % 64) % 64;
  constexpr int TILE = CO * CS;
  constexpr int NV4 = CO * W1 * 4;
  constexpr int PF = (NV4 + NTM - 1) / NTM;
  constexpr int RSL = S > K - S ? S : K - S;      // rows per stage (max)
  constexpr int CS1 = W0 * 16 + (80 - (W0 * 16) % 64) % 64;  // ring: channel stride
  constexpr int ROWF = CI * CS1;                 // ring: one row over g^(1), [CI][W0][16 q]
  constexpr int SLOT = RSL * ROWF;
  constexpr int PB = 2 * 4 * RSL * CI * W0;      // parameters: [2 sub-domains][4][RSL][CI][W0]
  constexpr int NPV4 = PB / 4;
  constexpr int PP = (NPV4 + NTM - 1) / NTM;
  extern __shared__ float lds[];
  float* tiles = lds;                // 2 x TILE
  float* ring = tiles + 2 * TILE;    // 3 x SLOT
  float* pars = ring + 3 * SLOT;     // 2 x PB
  float* red = pars + 2 * PB;        // (NS + C0) x 16

  const int lane = threadIdx.x & 63, wave = wave_id();
  const unsigned q0 = xcd_tile(blockIdx.x) * 16u;
  if (q0 >= Q) return;  // grid padding, uniform per block
  const unsigned R = (unsigned)s.R;
  const unsigned b0 = q0 / R;
  const unsigned b1 = (min(q0 + 15u, Q - 1u)) / R;  // b0 or b0 + 1
  auto yrow = [&](int e, int r) { return e < H1 ? e * S - P + r : (H1 - 1) * S - P + S + r; };
  auto nrows = [&](int e) { return e < H1 ? S : K - S; };
  constexpr int NSTEP = H1 + 3;

  if (wave < NM) {
    // ------------------------------------------------------------------ matrix waves
    const int n = lane & 15, G = lane >> 4;
    const int tid = threadIdx.x;
    float wreg[PER][KS];
    {
      const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
      for (int ph = 0; ph < PER; ++ph) {
        const int ky = ((slot - ph * S) % K + K) % K;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int co = 4 * ks + G;
          wreg[ph][ks] = (slot < K && kx < K) ? t.W[((co * CI + wave) * K + ky) * K + kx] : 0.f;
        }
      }
    }
    auto gaddr = [&](int y1, int v4) {
      const int cx = v4 >> 2, j4 = v4 & 3;
      const int co = cx / W1, x1 = cx - co * W1;
      return in + ((unsigned)(co * H1 + y1) * W1 + x1) * ldq + q0 + j4 * 4;
    };
    auto loff = [&](int v4) {
      const int cx = v4 >> 2, j4 = v4 & 3;
      const int co = cx / W1, x1 = cx - co * W1;
      return co * CS + x1 * 16 + j4 * 4;
    };
    auto pload = [&](int e, int v, float4v& out) {
      const int x4 = v % (W0 / 4);
      const int c = (v / (W0 / 4)) % CI;
      const int r = (v / (W0 / 4 * CI)) % RSL;
      const int arr = (v / (W0 / 4 * CI * RSL)) % 4;
      const int bsel = v / (W0 / 4 * CI * RSL * 4);
      const int y = yrow(e, r);
      out = float4v{0.f, 0.f, 0.f, 0.f};
      if (r >= nrows(e) || y < 0 || y >= H0 || b0 + bsel > b1) return;
      const unsigned rowi = ((unsigned)c * H0 + y) * W0 + 4 * x4;
      const long pb = (long)(b0 + bsel) * s.pstride + rowi;
      const float* src = arr == 0 ? s.a_lo + pb : arr == 1 ? s.a_up + pb
                       : arr == 2 ? s.b_up + pb : s.bias + rowi;
      out = *reinterpret_cast<const float4v*>(src);
    };
    auto park = [&](int t_, int r, const float* v) {
      float* dst = ring + (t_ % 3) * SLOT + r * ROWF + wave * CS1 + n;
#pragma unroll
      for (int x = 0; x < W0; ++x) dst[x * 16] = v[x];
    };

    for (int v4 = tid; v4 < NV4; v4 += NTM)
      *reinterpret_cast<float4v*>(tiles + loff(v4)) =
          *reinterpret_cast<const float4v*>(gaddr(0, v4));
    lds_barrier();

    float acc[W0];
#pragma unroll
    for (int x = 0; x < W0; ++x) acc[x] = 0.f;

    for (int ybase = 0; ybase < H1; ybase += PER) {
#pragma unroll
      for (int ph = 0; ph < PER; ++ph) {
        const int y1 = ybase + ph;
        if (H1 % PER != 0 && y1 >= H1) break;
        const float* tile = tiles + (y1 & 1) * TILE;
        const bool more = y1 + 1 < H1;
        float4v pf[PF], pp[PP];
#pragma unroll
        for (int k = 0; k < PF; ++k) {
          const int v4 = min(tid + k * NTM, NV4 - 1);
          pf[k] = *reinterpret_cast<const float4v*>(gaddr(more ? y1 + 1 : y1, v4));
        }
#pragma unroll
        for (int k = 0; k < PP; ++k) pload(y1, min(tid + k * NTM, NPV4 - 1), pp[k]);
#pragma unroll
        for (int x1 = 0; x1 < W1; ++x1) {
          float bv[KS];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) bv[ks] = tile[(4 * ks + G) * CS + x1 * 16 + n];
          float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ph][ks], bv[ks], d, 0, 0, 0);
#pragma unroll
          for (int kx = 0; kx < K; ++kx) {
            const int col = x1 * S - P + kx;
            if (col >= 0 && col < W0) acc[col] += d[kx];
          }
        }
        if (more) {
          float* nt = tiles + ((y1 + 1) & 1) * TILE;
#pragma unroll
          for (int k = 0; k < PF; ++k) {
            const int v4 = tid + k * NTM;
            if (v4 < NV4) *reinterpret_cast<float4v*>(nt + loff(v4)) = pf[k];
          }
        }
#pragma unroll
        for (int k = 0; k < PP; ++k) {
          const int v = tid + k * NTM;
          if (v < NPV4) *reinterpret_cast<float4v*>(pars + (y1 & 1) * PB + 4 * v) = pp[k];
        }
        const int ky = ((G - ph * S) % K + K) % K;
        if (G < K && ky < S) {
          park(y1, ky, acc);
#pragma unroll
          for (int x = 0; x < W0; ++x) acc[x] = 0.f;
        }
        lds_barrier();
      }
    }
    {  // step H1: the rows still open, and their parameters
      float4v pp[PP];
#pragma unroll
      for (int k = 0; k < PP; ++k) pload(H1, min(tid + k * NTM, NPV4 - 1), pp[k]);
      constexpr int ph_last = (H1 - 1) % PER;
      const int ky = ((G - ph_last * S) % K + K) % K;
      if (G < K && ky >= S) park(H1, ky - S, acc);
#pragma unroll
      for (int k = 0; k < PP; ++k) {
        const int v = tid + k * NTM;
        if (v < NPV4) *reinterpret_cast<float4v*>(pars + (H1 & 1) * PB + 4 * v) = pp[k];
      }
    }
    for (int st = H1; st < NSTEP; ++st) lds_barrier();
    lds_barrier();  // final reduction
    return;
  }

  if (wave < NM + NS) {
    // ------------------------------------------------------------------ storer waves
    const int ws = wave - NM;
    const int qn = lane & 15, xg = lane >> 4;
    const unsigned q = q0 + qn;
    const bool qok = q < Q;
    const int bsel = qok ? (int)(q / R - b0) : 0;
    float beta = 0.f;
    auto stage = [&](int e) {
      float* slot = ring + (e % 3) * SLOT;
      const float* pslot = pars + (e & 1) * PB;
      const int nr = nrows(e);
      for (int it = ws; it < nr * CI; it += NS) {
        const int r = it / CI, c = it - r * CI;
        const int y = yrow(e, r);
        if (y < 0 || y >= H0) continue;
        float* row = slot + r * ROWF + c * CS1 + qn;
        constexpr int AST = RSL * CI * W0;
        const float* pbase = pslot + ((bsel * 4) * RSL + r) * CI * W0 + c * W0 + 4 * xg;
        const float4v lo = *reinterpret_cast<const float4v*>(pbase);
        const float4v up = *reinterpret_cast<const float4v*>(pbase + AST);
        const float4v bu = *reinterpret_cast<const float4v*>(pbase + 2 * AST);
        const float4v bz = *reinterpret_cast<const float4v*>(pbase + 3 * AST);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int x = 4 * xg + j;
          const float a = row[x * 16];
          const bool pos = a >= 0.f;
          const float ah = a * (pos ? lo[j] : up[j]);
          if (qok) {
            beta = fmaf(pos ? 0.f : a, bu[j], beta);
            beta = fmaf(ah, bz[j], beta);
          }
          row[x * 16] = ah;
        }
      }
    };
    lds_barrier();  // initial tile
    for (int st = 0; st < NSTEP; ++st) {
      if (st >= 1 && st <= H1 + 1) stage(st - 1);
      lds_barrier();
    }
    beta += __shfl_xor(beta, 16, 64);
    beta += __shfl_xor(beta, 32, 64);
    if (lane < 16) red[ws * 16 + lane] = beta;
    lds_barrier();
    return;
  }

  // ---------------------------------------------------------------------- x waves
  const int xw = wave - NM - NS;  // input channel c0 of T_1
  const int n = lane & 15, G = lane >> 4;
  float wreg1[PER1][KS1];
  {
    const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
    for (int ph = 0; ph < PER1; ++ph) {
      const int ky = ((slot - ph * S1) % K1 + K1) % K1;
#pragma unroll
      for (int ks = 0; ks < KS1; ++ks) {
        const int c1 = 4 * ks + G;
        wreg1[ph][ks] = (slot < K1 && kx < K1) ? t1.W[((c1 * C0 + xw) * K1 + ky) * K1 + kx]
                                               : 0.f;
      }
    }
  }
  float acc1[WX];
#pragma unroll
  for (int x = 0; x < WX; ++x) acc1[x] = 0.f;
  float l1 = 0.f;
  auto emit = [&](int yx) {  // output row yx of channel xw: ||.||_1 over the image
    if (yx < 0 || yx >= HX) return;
#pragma unroll
    for (int x = 0; x < WX; ++x) l1 += fabsf(acc1[x]);
  };
  // T_1^T over one row y of g^(1), held in `row` ([CI][W0][16 q] with channel stride CS1)
  auto consume = [&](const float* row, int y) {
    const int ph = y % PER1;
    float wa[KS1];
#pragma unroll
    for (int ks = 0; ks < KS1; ++ks) {
      wa[ks] = wreg1[0][ks];
#pragma unroll
      for (int p2 = 1; p2 < PER1; ++p2)
        if (ph == p2) wa[ks] = wreg1[p2][ks];
    }
#pragma unroll
    for (int x1 = 0; x1 < W0; ++x1) {
      float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS1; ++ks)
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[ks], row[(4 * ks + G) * CS1 + x1 * 16 + n],
                                                d, 0, 0, 0);
#pragma unroll
      for (int kx = 0; kx < K1; ++kx) {
        const int col = x1 * S1 - P1 + kx;
        if (col >= 0 && col < WX) acc1[col] += d[kx];
      }
    }
    const int ky = ((G - ph * S1) % K1 + K1) % K1;
    if (G < K1 && ky < S1) {
      emit(y * S1 - P1 + ky);
#pragma unroll
      for (int x = 0; x < WX; ++x) acc1[x] = 0.f;
    }
  };
  lds_barrier();  // initial tile
  for (int st = 0; st < NSTEP; ++st) {
    if (st >= 2) {
      const int e = st - 2;
      const float* slot = ring + (e % 3) * SLOT;
      const int nr = nrows(e);
      for (int r = 0; r < nr; ++r) {
        const int y = yrow(e, r);
        if (y >= 0 && y < H0) consume(slot + r * ROWF, y);
      }
    }
    lds_barrier();
  }
  {  // output rows still open after the last row of g^(1)
    const int ph = (H0 - 1) % PER1;
    const int ky = ((G - ph * S1) % K1 + K1) % K1;
    if (G < K1 && ky >= S1) emit((H0 - 1) * S1 - P1 + ky);
  }
  l1 += __shfl_xor(l1, 16, 64);
  l1 += __shfl_xor(l1, 32, 64);
  if (lane < 16) red[(NS + xw) * 16 + lane] = l1;
  lds_barrier();
  if (xw != 0 || lane >= 16) return;
  const unsigned q = q0 + lane;
  if (q >= Q) return;
  float tb = 0.f, ta = 0.f;
  for (int w = 0; w < NS; ++w) tb += red[w * 16 + lane];
  for (int w = 0; w < C0; ++w) ta += red[(NS + w) * 16 + lane];
  Acc a{tb, 0.f, ta};
  sink_finish<MODE_BOUND>(s, a, q, q / R, q % R, false);
}

// The last two backward stages of a pass, T_2^T (Eq. 7) with the relaxation of layer 1 and
// T_1^T with the concretisation (Eq. 8), in one kernel, 16 rows per block, for two sources of
// the rows over g^(2):
//   FC: pass k opens at the fully connected layer k = 3 (rows +-e_j over h^(3)); the rows are
//     built from W_3 and relaxed onto layer 2 (Eq. 4, 6) as in k_convT_relax_ws, so nothing
//     but the bounds reaches global memory;
//   slab: the rows, already relaxed onto layer 2, are read from a slab [n_2][ldq] (the final
//     pass), and their running bias from Sink::beta.
// A block's rows span at most NBS sub-domains.  Wave roles, stepping through the same barriers:
//   matrix waves (CPW channels of g^(1) each): at step y1 they build (FC) or load (slab) the
//     input tile of row y1 + 1, run T_2^T on row y1, park the
//     rows over g^(1) that row completes ("stage y1"; stage H1 = the rows still open after the
//     last input row), unrelaxed, in slot y1 & 1 of an LDS ring, and stage the layer-1
//     relaxation of those rows beside them; every global load is theirs;
//   x waves (NXW of them, each owning a range of output columns of T_1^T over every input
//     channel): at step e + 1 they relax the rows of stage e as they read them (Eq. 6, each
//     entry once per wave that reads it, its intercept and bias terms added by one of them)
//     and carry them through T_1^T with the rotating lane-group scheme, one MFMA chain per
//     input channel of T_1 on the same relaxed operand, accumulating ||A_x||_1 per row.
//     Neighbouring column ranges share one input column (their borders are placed so), and
//     with NXW = NM each SIMD holds one wave of either role.
// The bound of a row is then its bias terms minus eps ||A_x||_1 (the linear term sits in the
// layer-1 bias).
// TAPE (FC source, for the reverse sweep): the matrix waves also store each parked row over
// g^(1), unrelaxed, to Sink::tape, and the x waves the sign of each entry of A_x to Sink::tsign,
// both blocked by groups of 8 rows, [q / 8][entry][q % 8], so that the reverse sweep, which
// takes 8 rows at a time, reads contiguous memory (rows past Q included: they lie inside the
// padded width ldq, and hold zeros).
template <int K, int S, int P, int H1, int W1, int H0, int W0, int CO, int CI, int CPW, int K1,
          int S1, int P1, int HX, int WX, int C0, int NXW, bool FC, int NBS, int SPEC = 0,
          bool TAPE = false>
__global__ void __launch_bounds__(64 * (CI / CPW + NXW))
__attribute__((amdgpu_waves_per_eu(SPEC > 0 ? 2 : (CI / CPW + NXW <= 8 ? 4 : 3), 8)))
    k_convT_fc_bound(DLayer t, DLayer t1, const float* __restrict__ in, unsigned ldq, unsigned Q,
                     Sink s, FcSrc fc) {
  static_assert(W0 == 16 && K <= 4 && S <= K && CO % 4 == 0 && CI % 4 == 0 && CI % CPW == 0,
                "geometry");
  static_assert(K1 <= 4 && S1 <= K1 && W1 % 4 == 0, "geometry");
  static_assert((H1 - 1) * S - P + K >= H0, "every output row is reached by an input row");
  static_assert((W1 - 1) * S - P + K >= W0 && P < K, "every output column is reached");
  static_assert((H0 - 1) * S1 - P1 + K1 >= HX, "every input row of T_1 is reached");
  constexpr int NM = CI / CPW;                   // matrix waves
  constexpr int NTM = 64 * NM;
  constexpr int KS = CO / 4, KS1 = CI / 4;
  constexpr int PER = (K % S == 0) ? K / S : K;
  constexpr int PER1 = (K1 % S1 == 0) ? K1 / S1 : K1;
  constexpr int TILE = W1 * CO * 16;             // input tile [W1][CO][16 q]
  constexpr int RSL = S > K - S ? S : K - S;     // rows over g^(1) per stage (max)
  // ring: a row over g^(1) is [CI][W0][16 q] with channel stride CS1; the pads put the four
  // lane groups of an x-wave read, and the two rows of a park, on different banks
  constexpr int CS1 = W0 * 16 + 16;
  constexpr int ROWF = CI * CS1 + 32;
  constexpr int SLOT = RSL * ROWF;
  // layer-1 relaxation of a stage, float4 (a_lo, a_up, b_up, z1) per entry:
  // [NBS sub-domains][RSL][CI][W0 (+1 pad)]
  static_assert(NBS == 2 || NBS == 3, "sub-domains per block");
  static_assert(SPEC == 0 || !FC, "the spec source replaces the slab source");
  static_assert(!TAPE || FC, "tapes are written for the FC source only");
  constexpr int NMT_S = CO * W1 / 16;  // spec source: 16-entry tiles of an input row
  static_assert(SPEC == 0 || (NMT_S % (CI / CPW) == 0 && W1 % 4 == 0), "spec tiles per wave");
  static_assert(SPEC == 0 || NMT_S / (CI / CPW) <= 2, "spec operands: two tiles per wave");
  constexpr int TPW_S = SPEC > 0 ? NMT_S / (CI / CPW) : 1;
  constexpr int PCS4 = W0 + 1;
  constexpr int PBS4 = RSL * CI * PCS4 + 2;
  constexpr int PSLOT4 = NBS * PBS4;
  constexpr int NPE = NBS * RSL * CI * W0;       // entries staged per stage
  constexpr int PL = (NPE + NTM - 1) / NTM;
  constexpr int NTASK = CO * W1 / 4 * 8;         // FC source tasks per input row
  constexpr int TPL = FC ? (NTASK + NTM - 1) / NTM : 1;
  constexpr int NV4 = CO * W1 * 4;               // slab source: float4 per input tile
  constexpr int PF = FC ? 1 : (NV4 + NTM - 1) / NTM;
  constexpr int NSTEP = H1 + 2;
  __shared__ float tiles[2][TILE];
  __shared__ float ring[2][SLOT];
  __shared__ float4v pars[2][PSLOT4];
  __shared__ float red[NM * 16 + 2 * NXW * 16];
  // spec source: the block's rows relaxed onto layer L-1, the MFMA B operand [4 SPEC][16 rows]
  __shared__ float vts[SPEC > 0 ? SPEC * 64 : 1];
  // border exchange of the x waves (see there): [step parity][wave - 1][channel, column][lane]
  constexpr int NSH = K1 - S1;  // output columns two neighbouring x waves share
  __shared__ float xb[2][NXW > 1 ? NXW - 1 : 1][C0 * NSH][64];

  const int lane = threadIdx.x & 63, wave = wave_id();
  const unsigned q0 = xcd_range(blockIdx.x) * 16u;
  if (q0 >= Q) return;  // grid padding, uniform per block
  const unsigned R = (unsigned)s.R;
  const unsigned b0 = q0 / R;
  const unsigned b1 = (min(q0 + 15u, Q - 1u)) / R;  // b1 - b0 < NBS
  auto yrow = [&](int e, int r) { return e < H1 ? e * S - P + r : (H1 - 1) * S - P + S + r; };
  auto nrows = [&](int e) { return e < H1 ? S : K - S; };

  if (wave < NM) {
    // ------------------------------------------------------------------ matrix waves
    const int n = lane & 15, G = lane >> 4;
    const int tid = threadIdx.x;  // < NTM
    float wreg[PER][CPW][KS];
    {
      const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
      for (int ph = 0; ph < PER; ++ph) {
        const int ky = ((slot - ph * S) % K + K) % K;
#pragma unroll
        for (int c = 0; c < CPW; ++c)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const int co = 4 * ks + G, ci = wave * CPW + c;
            wreg[ph][c][ks] = (slot < K && kx < K)
                                  ? t.W[((co * CI + ci) * K + ky) * K + kx] : 0.f;
          }
      }
    }
    auto park = [&](int e, int r, int c, const float* v) {
      float* dst = ring[e & 1] + r * ROWF + (wave * CPW + c) * CS1 + n;
#pragma unroll
      for (int x = 0; x < W0; ++x) dst[x * 16] = v[x];
      if constexpr (TAPE) {
        // buffer stores: a block-uniform base (the channel's plane in the block's first group
        // of 8 rows), the lane's row group, row and map row as the lane offset, the column as
        // the scalar offset
        const int y = yrow(e, r);
        if (y >= 0 && y < H0) {
          constexpr unsigned NG = CI * H0 * W0 * 8;  // floats of one group of 8 rows
          float* plane = s.tape + (size_t)(q0 >> 3) * NG + (size_t)(wave * CPW + c) * (H0 * W0 * 8);
          const unsigned boff =
              ((unsigned)(n >> 3) * NG + (unsigned)(n & 7) + (unsigned)y * (W0 * 8)) * 4u;
#pragma unroll
          for (int x = 0; x < W0; ++x) {
            const __amdgpu_buffer_rsrc_t rs =
                __builtin_amdgcn_make_buffer_rsrc(plane, (short)0, 0x7fffffff, 0x00020000);
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v[x]), rs, boff,
                                                  (unsigned)x * 32u, 0);
          }
        }
      }
    };
    // layer-1 relaxation of stage e: loaded into registers at the start of step e, written to
    // pars[e & 1] at its end.  Entries of rows outside the map or of a second sub-domain the
    // block does not have are never read: they load a clamped entry instead, so that the loads
    // carry no condition (a conditional value would make the wave wait for them at once).
    float4v pv[PL];
    auto pl_load = [&](int e) {
#pragma unroll
      for (int k = 0; k < PL; ++k) {
        const int v = min(tid + k * NTM, NPE - 1);
        const int x = v % W0, c = (v / W0) % CI, r = (v / (W0 * CI)) % RSL;
        const unsigned b = min(b0 + (unsigned)(v / (W0 * CI * RSL)), b1);
        const int y = min(max(yrow(e, r), 0), H0 - 1);
        const unsigned i = ((unsigned)c * H0 + y) * W0 + x;
        const unsigned pb = b * (unsigned)s.pstride + i;
        pv[k] = float4v{s.a_lo[pb], s.a_up[pb], s.b_up[pb], s.bias[i]};
      }
    };
    auto pl_store = [&](int e) {
#pragma unroll
      for (int k = 0; k < PL; ++k) {
        const int v = tid + k * NTM;
        const int x = v % W0, c = (v / W0) % CI, r = (v / (W0 * CI)) % RSL;
        const int bsel = v / (W0 * CI * RSL);
        if (v < NPE) pars[e & 1][bsel * PBS4 + (r * CI + c) * PCS4 + x] = pv[k];
      }
    };

    // FC source (as in k_convT_relax_ws): task tk of an input row = (quad qd of four
    // consecutive x1 of channel co, pair of rows q0 + 2 qp, q0 + 2 qp + 1)
    typedef float float2v __attribute__((ext_vector_type(2)));
    unsigned g_wa[TPL], g_wb[TPL], g_pb[TPL];
    float g_sa[TPL], g_sb[TPL], g_bz[TPL];
    int g_lds[TPL];
    bool g_on[TPL];
    float4v g_xa[TPL], g_xb[TPL], g_lo[TPL], g_up[TPL], g_bu[TPL];
    float fbeta_a = 0.f, fbeta_b = 0.f;
    if constexpr (FC) {
      const unsigned nin = CO * H1 * W1, nk = (unsigned)fc.nk;
#pragma unroll
      for (int k = 0; k < TPL; ++k) {
        const int tk = tid + k * NTM;
        g_on[k] = tk < NTASK;
        const int qp = tk & 7, qd = g_on[k] ? tk >> 3 : 0;
        const int co = qd % CO, t4 = qd / CO;
        const unsigned qa = q0 + 2u * qp, qb = qa + 1u;
        const unsigned ra = qa % R;
        // rows 2 qp, 2 qp + 1 are +e_j, -e_j of one neuron j (R is even): one row of W_k
        (void)nk;
        g_sa[k] = qa < Q ? 1.f : 0.f;
        g_sb[k] = qb < Q ? -1.f : 0.f;
        const unsigned i0 = (unsigned)co * H1 * W1 + 4u * t4;
        g_wa[k] = (ra >> 1) * nin + i0;
        g_wb[k] = g_wa[k];
        // R is even, so rows 2 qp and 2 qp + 1 share their sub-domain
        g_pb[k] = (qa < Q ? qa / R : b0) * (unsigned)s.pstride + i0;
        g_bz[k] = t.b[co];
        g_lds[k] = (4 * t4 * CO + co) * 16 + 2 * qp;
      }
    }
    auto gen_load = [&](int yg) {
#pragma unroll
      for (int k = 0; k < TPL; ++k)
        if (g_on[k]) {
          const unsigned o = (unsigned)yg * W1;
          g_xa[k] = *reinterpret_cast<const float4v*>(fc.W + (g_wa[k] + o));
          g_xb[k] = g_xa[k];
          g_lo[k] = *reinterpret_cast<const float4v*>(fc.a_lo + (g_pb[k] + o));
          g_up[k] = *reinterpret_cast<const float4v*>(fc.a_up + (g_pb[k] + o));
          g_bu[k] = *reinterpret_cast<const float4v*>(fc.b_up + (g_pb[k] + o));
        }
    };
    auto gen_store = [&](float* buf) {
#pragma unroll
      for (int k = 0; k < TPL; ++k)
        if (g_on[k]) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float a = g_sa[k] * g_xa[k][e], b = g_sb[k] * g_xb[k][e];
            const float ha = a * (a >= 0.f ? g_lo[k][e] : g_up[k][e]);
            const float hb = b * (b >= 0.f ? g_lo[k][e] : g_up[k][e]);
            fbeta_a = fmaf(fminf(a, 0.f), g_bu[k][e], fbeta_a);
            fbeta_a = fmaf(ha, g_bz[k], fbeta_a);
            fbeta_b = fmaf(fminf(b, 0.f), g_bu[k][e], fbeta_b);
            fbeta_b = fmaf(hb, g_bz[k], fbeta_b);
            *reinterpret_cast<float2v*>(buf + g_lds[k] + e * CO * 16) = float2v{ha, hb};
          }
        }
    };

    // slab source: float4 v of input row y1 (channel co, column x1, four rows q) to registers,
    // then to the tile
    float4v sv[PF];
    auto slab_load = [&](int y1) {
#pragma unroll
      for (int k = 0; k < PF; ++k) {
        const int v4 = min(tid + k * NTM, NV4 - 1);
        const int cx = v4 >> 2, j4 = v4 & 3;
        const int x1 = cx / CO, co = cx - x1 * CO;
        sv[k] = *reinterpret_cast<const float4v*>(
            in + (size_t)((unsigned)(co * H1 + y1) * W1 + x1) * ldq + q0 + j4 * 4);
      }
    };
    auto slab_store = [&](float* buf) {
#pragma unroll
      for (int k = 0; k < PF; ++k) {
        const int v4 = tid + k * NTM;
        if (v4 < NV4) *reinterpret_cast<float4v*>(buf + 4 * v4) = sv[k];
      }
    };
    // Spec source (final pass, rows q = (b, s) of the spec merged into the last layer): the
    // row over g^(L-1) is C_s W_L relaxed onto layer L-1 (Eq. 6), built once per wave in LDS;
    // each input row of T_2^T (entries (co, y1, x1) of g^(L-2)) is that row through W_{L-1}^T
    // on MFMA (M = 16 entries, K = 4 features j, N = 16 rows; TPW_S entry tiles per wave, their
    // operands loaded at the start of the step) relaxed onto layer L-2 into the input tile.
    // The rows' intercept and bias terms of both relaxations, and C_s b_L, go to sbeta.
    float sbeta = 0.f;
    float sa[SPEC > 0 ? SPEC : 1];  // the first tile's A operands, loaded a step ahead
    int spec_y1 = 0;                // the input row they belong to
    const unsigned qs = min(q0 + (unsigned)n, Q - 1u);  // this lane's row (clamped)
    const unsigned bs = qs / R;
    if constexpr (SPEC > 0) {
      // the matrix waves share the rows: wave w relaxes k-steps w, w + NM, ... (each feature
      // j once, its terms in the wave's sbeta); a barrier of both roles follows
      const int nj = fc.nk;
      const unsigned sn = qs - bs * R;
      const long pb3 = (long)bs * s.pstride;
#pragma unroll
      for (int t = 0; t < (SPEC + NM - 1) / NM; ++t) {
        const int k = wave + t * NM;
        if (k >= SPEC) break;  // uniform
        const int j = 4 * k + G;
        float ah = 0.f;
        if (j < nj) {
          // both slopes loaded, so that no load waits for the coefficient's sign
          const float a = fc.b[(long)sn * nj + j];
          const float lo = fc.r_lo[pb3 + j], up = fc.r_up[pb3 + j];
          ah = a * (a >= 0.f ? lo : up);
          sbeta = fmaf(fminf(a, 0.f), fc.r_bu[pb3 + j], sbeta);
          sbeta = fmaf(ah, fc.sbias_k1[j], sbeta);
        }
        vts[j * 16 + n] = ah;
      }
      if (wave == 0 && G == 0) sbeta += fc.b[(long)R * nj + sn];
      lds_barrier();  // the rows (matched by the x waves' first barrier of the spec source)
    }
    // A operands of entry tile mt of input row y1 (4 k + G < 4 (SPEC - 1) < nj for
    // k < SPEC - 1; the last k-step is clamped, its rows j >= nj meet zeros of the LDS rows)
    auto spec_a = [&](int mt, int y1, float* a) {
      const int nj = fc.nk, nin = CO * H1 * W1;
      const int e = mt * 16 + (lane & 15);  // A operand row: entry e = (co, x1)
      const int i = ((e / W1) * H1 + y1) * W1 + e % W1;
      const float* w = fc.W + (long)G * nin + i;
#pragma unroll
      for (int k = 0; k < SPEC - 1; ++k) a[k] = w[(long)4 * k * nin];
      a[SPEC - 1] = fc.W[(long)min(4 * (SPEC - 1) + G, nj - 1) * nin + i];
    };
    auto spec_load = [&](int y1) {
      if constexpr (SPEC > 0) {
        spec_a(wave, y1, sa);
        spec_y1 = y1;
      }
    };
    auto spec_store = [&](float* buf) {
      if constexpr (SPEC > 0) {
        const float* vt = vts;
        const long pb2 = (long)bs * s.pstride;
        float sb[SPEC];  // the other tiles' operands, loaded here
#pragma unroll
        for (int t = 0; t < TPW_S; ++t) {
          const int mt = wave + NM * t;
          if (t + 1 < TPW_S) spec_a(mt + NM, spec_y1, sb);
          // this lane's four D entries: consecutive x1 of one channel
          const int e0 = mt * 16 + 4 * G;
          const int i0 = ((e0 / W1) * H1 + spec_y1) * W1 + e0 % W1;
          const float4v p_lo = *reinterpret_cast<const float4v*>(fc.a_lo + pb2 + i0);
          const float4v p_up = *reinterpret_cast<const float4v*>(fc.a_up + pb2 + i0);
          const float4v p_bu = *reinterpret_cast<const float4v*>(fc.b_up + pb2 + i0);
          const float4v p_bz = *reinterpret_cast<const float4v*>(fc.sbias_k + i0);
          float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int k = 0; k < SPEC; ++k)
            d = __builtin_amdgcn_mfma_f32_16x16x4f32(t == 0 ? sa[k] : sb[k],
                                                     vt[(4 * k + G) * 16 + n], d, 0, 0, 0);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int e = mt * 16 + 4 * G + r;
            const float a = d[r];
            const float ah = a * (a >= 0.f ? p_lo[r] : p_up[r]);
            sbeta = fmaf(fminf(a, 0.f), p_bu[r], sbeta);
            sbeta = fmaf(ah, p_bz[r], sbeta);
            buf[((e % W1) * CO + e / W1) * 16 + n] = ah;
          }
        }
      }
    };
    auto src_load = [&](int y1) {
      if constexpr (SPEC > 0) spec_load(y1); else if constexpr (FC) gen_load(y1); else slab_load(y1);
    };
    auto src_store = [&](float* buf) {
      if constexpr (SPEC > 0) spec_store(buf); else if constexpr (FC) gen_store(buf); else slab_store(buf);
    };

    src_load(0);
    src_store(tiles[0]);
    lds_barrier();

    float acc[CPW][W0];
#pragma unroll
    for (int c = 0; c < CPW; ++c)
#pragma unroll
      for (int x = 0; x < W0; ++x) acc[c][x] = 0.f;

    for (int ybase = 0; ybase < H1; ybase += 2 * PER) {
#pragma unroll
      for (int u = 0; u < 2 * PER; ++u) {
        const int y1 = ybase + u;
        if (H1 % (2 * PER) != 0 && y1 >= H1) break;
        const int ph = u % PER;
        const float* tile = tiles[u & 1];
        pl_load(y1);
        if (y1 + 1 < H1) src_load(y1 + 1);
#pragma unroll
        for (int x1 = 0; x1 < W1; ++x1) {
          float bv[KS];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) bv[ks] = tile[(x1 * CO + 4 * ks + G) * 16 + n];
#pragma unroll
          for (int c = 0; c < CPW; ++c) {
            float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ph][c][ks], bv[ks], d, 0, 0, 0);
#pragma unroll
            for (int kx = 0; kx < K; ++kx) {
              const int col = x1 * S - P + kx;
              if (col >= 0 && col < W0) acc[c][col] += d[kx];
            }
          }
        }
        const int ky = ((G - ph * S) % K + K) % K;
        if (G < K && ky < S) {
#pragma unroll
          for (int c = 0; c < CPW; ++c) {
            park(y1, ky, c, acc[c]);
#pragma unroll
            for (int x = 0; x < W0; ++x) acc[c][x] = 0.f;
          }
        }
        if (y1 + 1 < H1) src_store(tiles[(u + 1) & 1]);
        pl_store(y1);
        lds_barrier();
      }
    }
    {  // step H1: the rows still open, and their relaxation
      pl_load(H1);
      constexpr int ph_last = (H1 - 1) % PER;
      const int ky = ((G - ph_last * S) % K + K) % K;
      if (G < K && ky >= S) {
#pragma unroll
        for (int c = 0; c < CPW; ++c) park(H1, ky - S, c, acc[c]);
      }
      pl_store(H1);
      lds_barrier();
    }
    lds_barrier();  // step H1 + 1
    if constexpr (FC) {
      // rows 2 qp, 2 qp + 1 of every task of this wave: lanes qp, qp + 8, ..., qp + 56
#pragma unroll
      for (int o = 8; o < 64; o <<= 1) {
        fbeta_a += __shfl_xor(fbeta_a, o, 64);
        fbeta_b += __shfl_xor(fbeta_b, o, 64);
      }
      if (lane < 8) {
        red[wave * 16 + 2 * lane] = fbeta_a;
        red[wave * 16 + 2 * lane + 1] = fbeta_b;
      }
    }
    if constexpr (SPEC > 0) {
      // row n's terms: lanes n, n + 16, n + 32, n + 48 of the wave
      sbeta += __shfl_xor(sbeta, 16, 64);
      sbeta += __shfl_xor(sbeta, 32, 64);
      if (lane < 16) red[wave * 16 + lane] = sbeta;
    }
    lds_barrier();  // the x waves' last border exchange
    lds_barrier();  // final reduction
    return;
  }

  // ---------------------------------------------------------------------- x waves
  static_assert(NXW >= 1 && NXW <= 4, "x waves");
  static_assert(W0 % NXW == 0 && NSH > 0, "x-wave column split");
  static_assert(S <= PER1 && K - S <= PER1, "at most one output row per lane and step");
  const int xw = wave - NM;
  const int n = lane & 15, G = lane >> 4;
  const unsigned q = q0 + n;
  const int bsel = q < Q ? (int)(q / R - b0) : 0;
  // the x waves carry the longer chain of each step: they go first when both roles can issue
  __builtin_amdgcn_s_setprio(2);
  // x wave j takes the input columns [j W0/NXW, (j+1) W0/NXW) of T_1^T (and adds their
  // intercept and bias terms).  Their image covers OW output columns from OL on; the first and
  // last NSH of them are shared with the neighbouring waves.  When a lane completes an output
  // row it adds |.| of its own columns to ||A_x||_1, publishes its partial sums of the left
  // shared columns in xb, and keeps those of the right ones; after the next barrier it adds
  // the right neighbour's published part to them and takes |.|.  A lane completes at most one
  // output row per step, so one pending row per lane suffices.  xw is made a constant so
  // that the column ranges are compile-time.
  auto xrun = [&](auto xb_) {
  constexpr int XB = decltype(xb_)::value;
  constexpr int NCX = W0 / NXW;
  constexpr int XL = XB * NCX, XH = XL + NCX - 1;
  constexpr int OL = XL * S1 - P1, OW = (NCX - 1) * S1 + K1;
  constexpr bool HASL = XB > 0, HASR = XB < NXW - 1;
  static_assert(2 * NSH <= OW, "shared columns");
  float wreg1[PER1][C0][KS1];
  {
    const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
    for (int ph = 0; ph < PER1; ++ph) {
      const int ky = ((slot - ph * S1) % K1 + K1) % K1;
#pragma unroll
      for (int c0 = 0; c0 < C0; ++c0)
#pragma unroll
        for (int ks = 0; ks < KS1; ++ks) {
          const int c1 = 4 * ks + G;
          wreg1[ph][c0][ks] = (slot < K1 && kx < K1)
                                  ? t1.W[((c1 * C0 + c0) * K1 + ky) * K1 + kx] : 0.f;
        }
    }
  }
  // The output columns (x1 - XL) S1 + kx of input column x1 do not overlap those of x1 + 2
  // (K1 = 2 S1), so each input column accumulates in place, as the MFMA's C operand, in one of
  // two families of float4 (x1 - XL even: ev, odd: od); a column of the output row is the sum
  // of its two family entries, formed when the row is emitted.
  static_assert(K1 == 2 * S1 && NCX % 2 == 0, "two column families");
  constexpr int NF = NCX / 2;
  float4v ev[C0][NF], od[C0][NF];
#pragma unroll
  for (int c0 = 0; c0 < C0; ++c0)
#pragma unroll
    for (int m = 0; m < NF; ++m) ev[c0][m] = od[c0][m] = float4v{0.f, 0.f, 0.f, 0.f};
  auto colv = [&](int c0, int x) {  // output column x (local) of channel c0
    float v = 0.f;
    if (x / K1 < NF) v = ev[c0][x / K1][x % K1];
    if (x >= S1 && (x - S1) / K1 < NF) v += od[c0][(x - S1) / K1][(x - S1) % K1];
    return v;
  };
  float l1 = 0.f, beta = 0.f;
  float pend[C0 * NSH];  // right shared columns of the pending row
  bool pend_ok = false;
  int pend_y = 0;
  // TAPE: the sign of entry (c0, yx, g) of this lane's row
  // (lane offset: the lane's row group and row and the row yx; the uniform part, channel and
  // column, goes in the scalar offset, so that no per-column address stays live in vector
  // registers)
  auto put_sign = [&](int c0, int yx, int g, float a) {
    if constexpr (TAPE) {
      constexpr unsigned NG = C0 * HX * WX * 8;  // bytes of one group of 8 rows
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          s.tsign + (size_t)(q0 >> 3) * NG, (short)0, 0x7fffffff, 0x00020000);
      const unsigned voff = (unsigned)(n >> 3) * NG + (unsigned)(n & 7) + (unsigned)(yx * WX * 8);
      const unsigned soff = (unsigned)(c0 * HX * WX + g) * 8u;
      __builtin_amdgcn_raw_buffer_store_b8((unsigned char)sign8(a), rs, voff, soff, 0);
    }
  };
  // output row yx completed by this lane (step parity par)
  auto emit = [&](int yx, int par) {
    const bool ok = yx >= 0 && yx < HX;
#pragma unroll
    for (int c0 = 0; c0 < C0; ++c0)
#pragma unroll
      for (int x = 0; x < OW; ++x) {
        const int g = OL + x;
        const bool left = HASL && x < NSH, right = HASR && x >= OW - NSH;
        const float a = colv(c0, x);
        if (!left && !right && g >= 0 && g < WX && ok) {
          l1 += fabsf(a);
          put_sign(c0, yx, g, a);
        }
        if (left) xb[par][XB - 1][c0 * NSH + x][lane] = a;
        if (right) pend[c0 * NSH + x - (OW - NSH)] = a;
      }
#pragma unroll
    for (int c0 = 0; c0 < C0; ++c0)
#pragma unroll
      for (int m = 0; m < NF; ++m) ev[c0][m] = od[c0][m] = float4v{0.f, 0.f, 0.f, 0.f};
    if (HASR) {
      pend_ok = ok;
      pend_y = yx;
    }
  };
  // the pending row of the previous step (parity par): add the right neighbour's part
  auto resolve = [&](int par) {
    if constexpr (HASR) {
      if (pend_ok) {
#pragma unroll
        for (int v = 0; v < C0 * NSH; ++v) {
          const float a = pend[v] + xb[par][XB][v][lane];
          l1 += fabsf(a);
          put_sign(v / NSH, pend_y, OL + OW - NSH + v % NSH, a);
        }
      }
      pend_ok = false;
    }
  };
  // relaxation and T_1^T of row y over g^(1): coefficients in `row`, relaxation in `prm`
  // ([CI][W0] float4 with channel stride PCS4, at this lane's sub-domain)
  // (phc: the phase y mod PER1 when it is a compile-time constant, else -1)
  auto consume = [&](const float* row, const float4v* prm, int y, int par, auto phc) {
    constexpr int PHC = decltype(phc)::value;
    const int ph = PHC >= 0 ? PHC : y % PER1;
    float wa[C0][KS1];
#pragma unroll
    for (int c0 = 0; c0 < C0; ++c0)
#pragma unroll
      for (int ks = 0; ks < KS1; ++ks) {
        if constexpr (PHC >= 0) {
          wa[c0][ks] = wreg1[PHC][c0][ks];
        } else {
          wa[c0][ks] = wreg1[0][c0][ks];
#pragma unroll
          for (int p2 = 1; p2 < PER1; ++p2)
            if (ph == p2) wa[c0][ks] = wreg1[p2][c0][ks];
        }
      }
    // Three columns in flight: the LDS reads of column x1 + 2 (into buffer x1 & 1), the MFMAs
    // of x1 and the relaxation of x1 + 1, whose reads were issued a column earlier.  The
    // scheduling barriers keep this order (and the compiler from reading further ahead); the
    // sums of column x1 are added one column later.
    float an[2][KS1], hn[KS1];
    float4v pn[2][KS1];
    auto fetch = [&](int x1) {
#pragma unroll
      for (int ks = 0; ks < KS1; ++ks) {
        const int c1 = 4 * ks + G;
        an[x1 & 1][ks] = row[c1 * CS1 + x1 * 16 + n];
        pn[x1 & 1][ks] = prm[c1 * PCS4 + x1];
      }
    };
    auto relax = [&](int x1) {
#pragma unroll
      for (int ks = 0; ks < KS1; ++ks) {
        const float a = an[x1 & 1][ks];
        const float4v p = pn[x1 & 1][ks];
        const float ah = a * (a >= 0.f ? p[0] : p[1]);
        beta = fmaf(fminf(a, 0.f), p[2], beta);
        beta = fmaf(ah, p[3], beta);
        hn[ks] = ah;
      }
    };
    fetch(XL);
    if (XL + 1 <= XH) fetch(XL + 1);
    relax(XL);
#pragma unroll
    for (int x1 = XL; x1 <= XH; ++x1) {
      if (x1 + 2 <= XH) fetch(x1 + 2);
      __builtin_amdgcn_sched_barrier(0);
      const int u = x1 - XL;
#pragma unroll
      for (int ks = 0; ks < KS1; ++ks)
#pragma unroll
        for (int c0 = 0; c0 < C0; ++c0) {
          float4v& a = (u % 2 == 0) ? ev[c0][u / 2] : od[c0][u / 2];
          a = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[c0][ks], hn[ks], a, 0, 0, 0);
        }
      if (x1 + 1 <= XH) relax(x1 + 1);
      __builtin_amdgcn_sched_barrier(0);
    }
    const int ky = ((G - ph * S1) % K1 + K1) % K1;
    if (G < K1 && ky < S1) emit(y * S1 - P1 + ky, par);
  };
  if constexpr (SPEC > 0) lds_barrier();  // the matrix waves' spec rows
  lds_barrier();  // first input tile
  for (int st = 0; st < NSTEP; ++st) {
    if (st >= 1) {
      resolve((st - 1) & 1);
      const int e = st - 1;
      const float* slot = ring[e & 1];
      const int nr = nrows(e);
      // row r of a step has y = (multiple of S) - P + r: its phase is fixed when PER1 | S
      auto row_r = [&](auto rc) {
        constexpr int r = decltype(rc)::value;
        constexpr int PHC = S % PER1 == 0 ? ((r - P) % PER1 + PER1) % PER1 : -1;
        const int y = yrow(e, r);
        if (r < nr && y >= 0 && y < H0)
          consume(slot + r * ROWF, pars[e & 1] + bsel * PBS4 + r * CI * PCS4, y, st & 1,
                  std::integral_constant<int, PHC>());
      };
      static_assert(RSL <= 4, "rows per step");
      row_r(std::integral_constant<int, 0>());
      if constexpr (RSL > 1) row_r(std::integral_constant<int, 1>());
      if constexpr (RSL > 2) row_r(std::integral_constant<int, 2>());
      if constexpr (RSL > 3) row_r(std::integral_constant<int, 3>());
    }
    lds_barrier();
  }
  resolve((NSTEP - 1) & 1);
  {  // output rows still open after the last row of g^(1)
    const int ph = (H0 - 1) % PER1;
    const int ky = ((G - ph * S1) % K1 + K1) % K1;
    if (G < K1 && ky >= S1) emit((H0 - 1) * S1 - P1 + ky, NSTEP & 1);
  }
  lds_barrier();
  resolve(NSTEP & 1);
  l1 += __shfl_xor(l1, 16, 64);
  l1 += __shfl_xor(l1, 32, 64);
  beta += __shfl_xor(beta, 16, 64);
  beta += __shfl_xor(beta, 32, 64);
  if (lane < 16) {
    red[NM * 16 + XB * 16 + lane] = beta;
    red[NM * 16 + (NXW + XB) * 16 + lane] = l1;
  }
  };
  if (xw == 0) xrun(std::integral_constant<int, 0>());
  if (NXW > 1 && xw == 1) xrun(std::integral_constant<int, (NXW > 1 ? 1 : 0)>());
  if (NXW > 2 && xw == 2) xrun(std::integral_constant<int, (NXW > 2 ? 2 : 0)>());
  if (NXW > 3 && xw == 3) xrun(std::integral_constant<int, (NXW > 3 ? 3 : 0)>());
  lds_barrier();
  if (xw != 0 || lane >= 16) return;
  // FC: the row's own bias +-b_k[j] and the terms of the relaxation onto layer 2 (slab: the
  // running bias, added by sink_finish); the terms of the relaxation onto layer 1
  const unsigned r = q % R;
  float tb = 0.f;
  if constexpr (FC) {
    const float bj = fc.b[(r >> 1) % (unsigned)fc.nk];
    tb = (r & 1) ? -bj : bj;
    for (int w = 0; w < NM; ++w) tb += red[w * 16 + lane];
  }
  if constexpr (SPEC > 0) {
    for (int w = 0; w < NM; ++w) tb += red[w * 16 + lane];
  }
  for (int w = 0; w < NXW; ++w) tb += red[NM * 16 + w * 16 + lane];
  float ta = 0.f;
  for (int w = 0; w < NXW; ++w) ta += red[NM * 16 + (NXW + w) * 16 + lane];
  if constexpr (FC) {
    // rows 2j, 2j + 1 (lanes 2i, 2i + 1) give l_j and -u_j; then the relaxation of layer k
    const float v = tb - s.eps * ta;
    const float vn = __shfl_xor(v, 1, 64);
    if (q >= Q || (r & 1)) return;  // (Q is even: row q + 1 exists)
    const unsigned b = q / R, jj = r >> 1;
    const long pi = (long)b * fc.n_relu + fc.off + jj;
    float lv = v, uv = -vn;
    parent_clip(lv, uv, fc.lpar, fc.upar, pi);
    s.lo[b * s.bstride + jj] = lv;
    s.hi[b * s.bstride + jj] = uv;
    const Relax1 rx = relax_neuron(lv, uv, fc.split ? fc.split[pi] : 0,
                                   fc.alpha ? fc.alpha + pi : nullptr);
    const long pp = (long)b * s.pstride + jj;
    fc.r_lo[pp] = rx.lo;
    fc.r_up[pp] = rx.up;
    fc.r_bu[pp] = rx.bu;
    fc.code[pi] = (int8_t)rx.code;
  } else {
    if (q >= Q) return;
    Acc a{tb, 0.f, ta};
    // (spec source: no running bias from an earlier stage)
    sink_finish<MODE_BOUND>(s, a, q, q / R, r, SPEC > 0);
  }
}

// The 16 rows +-e_j of a receptive-field block share the window (y2, x2) of one sub-domain:
// both signs of 8 consecutive output channels (block group g: channels 8g .. 8g + 7; row r:
// sign r / 8, channel 8g + r % 8), so rows r and r + 8 give l and u of one neuron.  C2 is a
// multiple of 8.  Blocks are ordered (sub-domain, group, y2, x2), x2 fastest.
__host__ __device__ constexpr int cgcd(int a, int b) { return b ? cgcd(b, a % b) : a; }

struct P2Row {
  int c2;
  bool neg;
};
__device__ __forceinline__ P2Row p2_row(int C2, int g, int r) {
  (void)C2;
  return {g * 8 + (r & 7), r >= 8};
}
__host__ __device__ inline int p2_groups(int C2) { return C2 / 8; }

// Pass 2 restricted to each row's receptive field, when T_2 and T_1 are convolutions.  (The
// kernel also writes the relaxation of layer 2, as k_relax_params would from its bounds.)
// Row +-e_j of h^(2), j = (c2, y2, x2), carried through T_2 is +-W_2[c2] placed on the window
// (y2*S2 - P2 + ky2, x2*S2 - P2 + kx2) of g^(1) and zero elsewhere, so its image under the
// relaxation of layer 1 and T_1^T is confined to that window's footprint on the input.  One
// block takes 16 rows that share a window -- one sub-domain, one sign, 16 consecutive c2 -- and
//  (1) writes their relaxed window coefficients to LDS (Eq. 6), accumulating the intercept and
//      layer-1 bias terms of each row in a fixed order,
//  (2) applies T_1^T to the window on 16x16x4 MFMA (one wave per input channel of T_1, the
//      same rotating lane-group scheme as k_convT_mfma), and
//  (3) concretises the footprint (Eq. 8; positions outside the image are zero padding) and
//      writes l_j (sign +) or u_j (sign -) of the sub-domain.
// The result equals the dense pass exactly in arithmetic terms: the skipped products are zeros.
template <int K1, int S1, int P1, int K2, int C1, int NW, int XW>
// (with 8 windows per block the kernel fits 80 VGPRs with 8 channels on T_1, 128 with 16, one
// more wave per SIMD than it would take unhinted; with 4 it would spill, so it is left alone)
__global__ void __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(XW == 8 ? (C1 >= 16 ? 4 : 6) : 1, 8)))
    k_pass2_window(DLayer t1, DLayer t2, long nb, const float* __restrict__ a_lo,
               const float* __restrict__ a_up, const float* __restrict__ b_up, long pstride,
               const float* __restrict__ z1, float eps, float* __restrict__ L,
               float* __restrict__ U, long n_relu, long off2, const int8_t* __restrict__ split,
               const float* __restrict__ alpha, float* __restrict__ lo2, float* __restrict__ up2,
               float* __restrict__ bu2, int8_t* __restrict__ code2, const float* __restrict__ lpar,
               const float* __restrict__ upar) {
  static_assert(C1 % 4 == 0 && K1 <= 4 && K2 <= 4, "unsupported geometry");
  constexpr int KS = C1 / 4;
  constexpr int NT = 64 * NW;
  constexpr int NPOS = K2 * K2;
  constexpr int NE = C1 * NPOS;                      // window entries per row
  constexpr int WO = (K2 - 1) * S1 + K1;           // footprint width on the input
  constexpr int PER = (K1 % S1 == 0) ? K1 / S1 : K1;
  constexpr int CS = NPOS * 16 + (80 - (NPOS * 16) % 64) % 64;  // channel stride, 16 mod 64
  constexpr int NEL = C1 * CS;                      // relaxed window tile
  constexpr int RPT = NT / 16;                      // threads per row in phase 1
  constexpr int NEP = (NE + RPT - 1) / RPT;         // window entries per thread (phase 1)
  constexpr int NPP = (NE + NT - 1) / NT;           // staged parameters per thread
  __shared__ float tile[NEL];
  __shared__ float red[NW * 16 + RPT * 16];
  __shared__ float4v prm[NE];  // (a_lo, a_up, b_up, W1 x0 + b1) of the window (0 outside)
  __shared__ float vb[XW][16];  // the rows' bounds, written out once per block
  float* bred = red + NW * 16;

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int n = lane & 15, G = lane >> 4;
  // block -> (sub-domain, row group, y2, XW consecutive windows along x2)
  const int H2 = t2.out_h, W2 = t2.out_w, C2 = t2.out_c;
  const int NG = p2_groups(C2);
  const int nxc = W2 / XW;
  unsigned blk = xcd_range(blockIdx.x);  // 32-bit: the scalar divisions stay short
  const int x2c = (int)(blk % (unsigned)nxc); blk /= (unsigned)nxc;
  const int y2 = (int)(blk % (unsigned)H2); blk /= (unsigned)H2;
  const int g = (int)(blk % (unsigned)NG); blk /= (unsigned)NG;
  const long b = blk;
  const int Y1 = y2 * t2.stride - t2.pad;  // window origin on g^(1), rows
  const int H1 = t1.out_h, Wd1 = t1.out_w;
  const long pb = b * pstride;

  // this thread's entries of W_2 (phase 1: row = tid mod 16, entries part, part + RPT, ...),
  // the same for every window of the block
  const int row = threadIdx.x & 15, part = threadIdx.x >> 4;
  const P2Row prw = p2_row(C2, g, row);
  const float sgn = prw.neg ? -1.f : 1.f;
  // split by sign (relaxed entry = wp a_lo + wn a_up), and the entry's place in the tile.
  // Entries k and k + TP lie TS channels apart at the same position, so only the first TP
  // places are held; the others are those plus a constant (an immediate LDS offset).
  constexpr int TP = NPOS / cgcd(RPT, NPOS), TS = TP * RPT / NPOS;
  float wp[NEP], wn[NEP];
  int toff[TP];
  {
    const float* w2 = t2.W + (long)prw.c2 * NE;  // [C1][K2][K2] of output channel c2
#pragma unroll
    for (int k = 0; k < NEP; ++k) {
      const int e = part + k * RPT;
      const float w = e < NE ? sgn * w2[e] : 0.f;
      wp[k] = fmaxf(w, 0.f);
      wn[k] = fminf(w, 0.f);
    }
#pragma unroll
    for (int k = 0; k < TP; ++k) {
      const int e = part + k * RPT;
      const int c1 = e / NPOS, pos = e - c1 * NPOS;
      toff[k] = c1 * CS + pos * 16 + row;
    }
  }
  // relaxation parameters of a window, one neuron per (thread, k)
  float4v pn[NPP];
  auto pfetch = [&](int X1) {
#pragma unroll
    for (int k = 0; k < NPP; ++k) {
      const int e = threadIdx.x + k * NT;
      pn[k] = float4v{0.f, 0.f, 0.f, 0.f};
      if (e >= NE) continue;
      const int c1 = e / NPOS, pos = e - c1 * NPOS;
      const int ky2 = pos / K2, kx2 = pos - ky2 * K2;
      const int y1 = Y1 + ky2, x1 = X1 + kx2;
      if (y1 >= 0 && y1 < H1 && x1 >= 0 && x1 < Wd1) {
        const long ni = ((long)c1 * H1 + y1) * Wd1 + x1;
        pn[k] = float4v{a_lo[pb + ni], a_up[pb + ni], b_up[pb + ni], z1[ni]};
      }
    }
  };

  // T_1^T weights, one wave per input channel c0 of T_1
  const int c0 = wave;
  const bool cok = c0 < t1.in_c;
  float wreg[PER][KS];
  {
    const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
    for (int ph = 0; ph < PER; ++ph) {
      const int ky = ((slot - ph * S1) % K1 + K1) % K1;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int c1 = 4 * ks + G;
        wreg[ph][ks] = (cok && slot < K1 && kx < K1)
                           ? t1.W[(((long)c1 * t1.in_c + c0) * K1 + ky) * K1 + kx] : 0.f;
      }
    }
  }
  const int Hi = t1.in_h, Wi = t1.in_w;
  const int OY = Y1 * S1 - P1;  // footprint origin on the input, rows

  pfetch(x2c * XW * t2.stride - t2.pad);
  for (int xi = 0; xi < XW; ++xi) {
    const int x2 = x2c * XW + xi;
    const int X1 = x2 * t2.stride - t2.pad;
    // (1) stage the window's parameters; fetch the next window's; relaxed coefficients of the
    // 16 rows and their bias terms
#pragma unroll
    for (int k = 0; k < NPP; ++k) {
      const int e = threadIdx.x + k * NT;
      if (e < NE) prm[e] = pn[k];
    }
    __syncthreads();
    if (xi + 1 < XW) pfetch(X1 + t2.stride);
    {
      float bpart = 0.f;
#pragma unroll
      for (int k = 0; k < NEP; ++k) {
        // (no early exit: the loop unrolls, so the arrays are indexed statically)
        const int e = part + k * RPT;
        if (k + 1 < NEP || e < NE) {  // (only the last k can fall past NE)
          const float4v pr = prm[e];
          const float v = fmaf(wp[k], pr[0], wn[k] * pr[1]);
          bpart = fmaf(wn[k], pr[2], bpart);
          // layer-1 bias and the linear term of the concretisation together: v (W1 x0 + b1)
          bpart = fmaf(v, pr[3], bpart);
          tile[toff[k % TP] + (k / TP) * TS * CS] = v;
        }
      }
      bred[part * 16 + row] = bpart;
    }
    __syncthreads();

    // (2) T_1^T on the window.  A lane's row of acc restarts after the lane emits it: the
    // first contribution of the next window row to each column then scales the old value by
    // keep = 0 (instead of clearing the row; every column is reached in every window row).
    const int OX = X1 * S1 - P1;
    float l1 = 0.f;
    float acc[WO];
    float keep = 1.f;
    const bool inside_x = OX >= 0 && OX + WO <= Wi;
    auto emit = [&](int yl) {  // local footprint row yl of channel c0: ||.||_1 of the clipped row
      const int y = OY + yl;
      if (!cok || y < 0 || y >= Hi) return;
      if (inside_x) {
#pragma unroll
        for (int x = 0; x < WO; ++x) l1 += fabsf(acc[x]);
      } else {
#pragma unroll
        for (int x = 0; x < WO; ++x) {
          const int xc = OX + x;
          l1 += (xc >= 0 && xc < Wi) ? fabsf(acc[x]) : 0.f;
        }
      }
    };
#pragma unroll
    for (int j = 0; j < K2; ++j) {
      const int ph = j % PER;
#pragma unroll
      for (int i = 0; i < K2; ++i) {
        const int pos = j * K2 + i;
        float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ph][ks],
                                                  tile[(4 * ks + G) * CS + pos * 16 + n], d,
                                                  0, 0, 0);
#pragma unroll
        for (int kx = 0; kx < K1; ++kx) {
          float& a = acc[i * S1 + kx];
          if (i > 0 && kx < K1 - S1)
            a += d[kx];
          else if (j == 0)
            a = d[kx];
          else
            a = fmaf(a, keep, d[kx]);
        }
      }
      const int ky = ((G - ph * S1) % K1 + K1) % K1;
      const bool done = G < K1 && ky < S1;
      if (done) emit(j * S1 + ky);
      keep = done ? 0.f : 1.f;
    }
    {
      const int ky = ((G - ((K2 - 1) % PER) * S1) % K1 + K1) % K1;
      if (G < K1 && ky >= S1) emit((K2 - 1) * S1 + ky);
    }

    // (3) reduce over lane groups and waves; add the bias terms; write the bound
    l1 += __shfl_xor(l1, 16, 64);
    l1 += __shfl_xor(l1, 32, 64);
    if (lane < 16) red[wave * 16 + lane] = l1;
    __syncthreads();
    if (threadIdx.x < 16) {
      const int r = threadIdx.x;
      const P2Row pr = p2_row(C2, g, r);
      float ta = 0.f, tb = (pr.neg ? -1.f : 1.f) * t2.b[pr.c2];
      for (int w = 0; w < NW; ++w) ta += red[w * 16 + r];
      for (int q = 0; q < RPT; ++q) tb += bred[q * 16 + r];
      vb[xi][r] = tb - eps * ta;
    }
  }
  // l and u of the block's 8 neurons in each of its XW windows (rows r and r + 8 are +-e_j of
  // one neuron), and their relaxation for the passes above: XW consecutive neurons per channel
  __syncthreads();
  if (threadIdx.x < 8 * XW) {
    const int cc = threadIdx.x / XW, xi = threadIdx.x - cc * XW;
    const long j = ((long)(g * 8 + cc) * H2 + y2) * W2 + x2c * XW + xi;
    const long pi = b * n_relu + off2 + j;
    float l = vb[xi][cc], u = -vb[xi][cc + 8];
    parent_clip(l, u, lpar, upar, pi);
    L[pi] = l;
    U[pi] = u;
    const Relax1 rx = relax_neuron(l, u, split ? split[pi] : 0, alpha ? alpha + pi : nullptr);
    lo2[b * pstride + j] = rx.lo;
    up2[b * pstride + j] = rx.up;
    bu2[b * pstride + j] = rx.bu;
    code2[pi] = (int8_t)rx.code;
  }
}

// LDS slot of channel c (0..7) in a tile the position-pair gather writes: bits 1 and 2 of c
// exchanged (an involution).  The gather's lane groups store channels c and c + 4 at two
// positions; with channel strides of 16 mod 64 banks, c and c + 4 would share banks, their
// slots lie two strides (32 banks) apart.
__host__ __device__ constexpr int slot8(int c) {
  return (c & ~6) | ((c & 2) << 1) | ((c & 4) >> 1);
}

// T^T of a stride-1 convolution (kernel KK <= 3, Cs source channels) as a gather onto a window
// of 8 destination channels, DW x DW positions, from a source window SW x SW: the 16 rows of a
// block are the N dimension, and the 16 M lanes take the 8 channels at two neighbouring
// positions (x0, x0 + 1) of a destination row, whose tap columns together span the four K
// lanes of a step (source column x0 + 1 - G for lane group G: tap G - 1 for x0, tap G for
// x0 + 1), so one MFMA serves both positions.  One K step per (source channel, tap row), the
// source row uniform (steps without one are skipped); position pairs are dealt to the waves.
// Each result is relaxed (Eq. 6) with pp[e] = (a_lo, a_up, b_up, bias), written to
// dst[slot8(c)][p][row], and its intercept and bias terms are summed into the returned value.
// Source and destination tiles: [channel slot][position][16 rows], channel strides SCS and DCS
// (16 mod 64 banks); the source's channels sit at slot8(c) when SRC_SLOT, else at c.
template <int Cs, int KK, int SW, int DW, int NW, bool SRC_SLOT>
__device__ __forceinline__ float gather_pair8(const float* __restrict__ W, const float* src,
                                              int SCS, float* dst, int DCS, const float4v* pp) {
  static_assert(KK <= 3, "two positions' tap columns fit the four K lanes");
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int n = lane & 15, G = lane >> 4;
  const int cm = n & 7, pm = n >> 3;  // A operand row: destination channel and position
  const int kx = G - 1 + pm;
  // (every lane loads from an in-range tap column, so the loads carry no branch; a lane whose
  // column lies outside the kernel then takes a zero weight)
  const bool kok = kx >= 0 && kx < KK;
  const float* wl = W + cm * KK * KK + min(max(kx, 0), KK - 1);
  float areg[Cs * KK];
#pragma unroll
  for (int ks = 0; ks < Cs * KK; ++ks) {
    const int c = ks / KK, ky = ks % KK;
    const float v = wl[(c * 8 * KK + ky) * KK];
    areg[ks] = kok ? v : 0.f;
  }
  constexpr int NP = (DW + 1) / 2;  // position pairs per destination row
  constexpr int ND = DW * DW;
  float bpart = 0.f;
  for (int pi = wave; pi < DW * NP; pi += NW) {
    const int y = pi / NP, x0 = 2 * (pi - y * NP);
    const int ix = x0 + 1 - G;
    const bool xok = ix >= 0 && ix < SW;
    const float* colp = src + (xok ? ix : 0) * 16 + n;
    float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ky = 0; ky < KK; ++ky) {
      const int iy = y - ky;
      if (iy < 0 || iy >= SW) continue;  // uniform
#pragma unroll
      for (int c = 0; c < Cs; ++c) {
        const float bv = xok ? colp[(SRC_SLOT ? slot8(c) : c) * SCS + iy * SW * 16] : 0.f;
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(areg[c * KK + ky], bv, d, 0, 0, 0);
      }
    }
    // lane (n, G) holds rows n of channels 4 (G & 1) + r at position x0 + (G >> 1)
    const int x = x0 + (G >> 1);
    if (x < DW) {
      const int p = y * DW + x;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = 4 * (G & 1) + r;
        const float4v q = pp[c * ND + p];
        const float a = d[r];
        const float ah = a >= 0.f ? a * q[0] : a * q[1];
        bpart = fmaf(fminf(a, 0.f), q[2], bpart);
        bpart = fmaf(ah, q[3], bpart);
        dst[slot8(c) * DCS + p * 16 + n] = ah;
      }
    }
  }
  return bpart;
}

// T_1^T over a W x W window tile of g^(1) ([channel slot][position][16 rows], 8 slots at
// stride CS, channel slot8(c) at slot c) for input channel c0 of T_1, with the rotating
// lane-group scheme of k_pass2_window, and the L1 norm of the result over the window's footprint
// on x (origin OY, OX; positions outside the image are zero padding): this lane's part of
// ||A_x||_1 of row n (Eq. 8).  A lane's row of acc restarts after the lane emits it: the next
// window row's first contribution to each column scales the old value by keep = 0 (every
// column is reached in every window row), and a footprint inside the image horizontally is
// summed without a per-column test.
template <int W, int K1, int S1, int KS, int CS>
__device__ __forceinline__ float t1t_window_l1(const DLayer& t1, int c0, const float* tile,
                                               int OY, int OX) {
  constexpr int PER = (K1 % S1 == 0) ? K1 / S1 : K1;
  constexpr int WO = (W - 1) * S1 + K1;  // footprint width on x
  const int lane = threadIdx.x & 63, n = lane & 15, G = lane >> 4;
  float wreg[PER][KS];
  {
    const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
    for (int ph = 0; ph < PER; ++ph) {
      const int ky = ((slot - ph * S1) % K1 + K1) % K1;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int c1 = slot8(4 * ks + G);  // (the tile holds channel slots)
        wreg[ph][ks] = (slot < K1 && kx < K1)
                           ? t1.W[(((long)c1 * t1.in_c + c0) * K1 + ky) * K1 + kx] : 0.f;
      }
    }
  }
  const int Hi = t1.in_h, Wi = t1.in_w;
  const bool inside_x = OX >= 0 && OX + WO <= Wi;
  float l1 = 0.f, keep = 1.f;
  float acc[WO];
  auto emit = [&](int yl) {  // footprint row yl: ||.||_1 of the clipped row
    const int y = OY + yl;
    if (y < 0 || y >= Hi) return;
    if (inside_x) {
#pragma unroll
      for (int x = 0; x < WO; ++x) l1 += fabsf(acc[x]);
    } else {
#pragma unroll
      for (int x = 0; x < WO; ++x) {
        const int xc = OX + x;
        l1 += (xc >= 0 && xc < Wi) ? fabsf(acc[x]) : 0.f;
      }
    }
  };
#pragma unroll
  for (int j = 0; j < W; ++j) {
    const int ph = j % PER;
#pragma unroll
    for (int i = 0; i < W; ++i) {
      const int pos = j * W + i;
      float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ph][ks],
                                                tile[(4 * ks + G) * CS + pos * 16 + n], d, 0,
                                                0, 0);
#pragma unroll
      for (int kx = 0; kx < K1; ++kx) {
        float& a = acc[i * S1 + kx];
        if (i > 0 && kx < K1 - S1)
          a += d[kx];
        else if (j == 0)
          a = d[kx];
        else
          a = fmaf(a, keep, d[kx]);
      }
    }
    const int ky = ((G - ph * S1) % K1 + K1) % K1;
    const bool done = G < K1 && ky < S1;
    if (done) emit(j * S1 + ky);
    keep = done ? 0.f : 1.f;
  }
  {
    const int ky = ((G - ((W - 1) % PER) * S1) % K1 + K1) % K1;
    if (G < K1 && ky >= S1) emit((W - 1) * S1 + ky);
  }
  return l1;
}

// Pass 3 restricted to each row's receptive field, when T_3, T_2 (stride 1) and T_1 are
// convolutions.  Row +-e_j of h^(3), j = (c3, y3, x3), carried through T_3 is +-W_3[c3] on the
// K3 x K3 window of j on g^(2); after the layer-2 relaxation, T_2^T spreads it over a
// (K3 + K2 - 1)^2 window of g^(1), and after the layer-1 relaxation T_1^T over that window's
// footprint on x.  One block of 8 waves takes the 16 rows sharing a window (rows as in
// k_pass2_window, over the channels of h^(3)):
//  (1) stages the relaxation parameters of both windows (zeros outside the maps),
//  (2) relaxes the g^(2) window (Eq. 6) with its intercept and bias terms,
//  (3) applies T_2^T as a gather on 16x16x4 MFMA (M = channels of g^(1), K = (c2, ky, kx)), one
//      g^(1) window position per wave at a time, and relaxes the result into an LDS tile,
//  (4) applies T_1^T to that tile with the rotating lane-group scheme (one wave per input
//      channel of T_1) and concretises (Eq. 8),
//  (5) writes l_j or u_j.  Arithmetically the dense pass minus products with zero.
template <int K3, int P3, int K2, int P2, int K1, int S1, int P1, int C1, int C2>
__global__ void __launch_bounds__(512)
    k_pass3_window(DLayer t1, DLayer t2, DLayer t3, const float* __restrict__ a_lo,
                   const float* __restrict__ a_up, const float* __restrict__ b_up, long pstride,
                   long poff1, long poff2, const float* __restrict__ bias, float eps,
                   float* __restrict__ L, float* __restrict__ U, long n_relu, long off3) {
  constexpr int NW = 8, NT = 64 * NW;
  constexpr int N2 = K3 * K3;               // g^(2) window positions
  constexpr int W1W = K3 - 1 + K2;          // g^(1) window width (T_2 has stride 1)
  constexpr int N1 = W1W * W1W;
  constexpr int E2 = C2 * N2, E1 = C1 * N1;
  constexpr int WO = (W1W - 1) * S1 + K1;   // footprint width on x
  constexpr int KS1 = C1 / 4;
  constexpr int PER1 = (K1 % S1 == 0) ? K1 / S1 : K1;
  constexpr int CS2 = N2 * 16 + (80 - (N2 * 16) % 64) % 64;
  constexpr int CS1 = N1 * 16 + (80 - (N1 * 16) % 64) % 64;
  constexpr int RP = NT / 16;               // threads per row in (2)
  static_assert(C1 % 4 == 0 && C1 <= 16 && K1 <= 4 && K2 <= 4 && K3 <= 4, "geometry");
  __shared__ float tile2[C2 * CS2];
  __shared__ float tile1[C1 * CS1];
  __shared__ float4v p2s[E2];  // (a_lo, a_up, b_up, bias) of the g^(2) window
  __shared__ float4v p1s[E1];  // (a_lo, a_up, b_up, W1 x0 + b1) of the g^(1) window
  __shared__ float rb2[RP * 16];  // bias terms of (2), per (part, row)
  __shared__ float rb1[NW * 4 * 16];  // bias terms of (3), per (wave, lane group, row)
  __shared__ float rl1[NW * 16];  // ||A_x||_1 partials of (4)

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int n = lane & 15, G = lane >> 4;
  const int H3 = t3.out_h, W3 = t3.out_w, C3 = t3.out_c;
  const int NG = p2_groups(C3);
  unsigned blk = xcd_range(blockIdx.x);  // 32-bit: the scalar divisions stay short
  const int x3 = (int)(blk % (unsigned)W3); blk /= (unsigned)W3;
  const int y3 = (int)(blk % (unsigned)H3); blk /= (unsigned)H3;
  const int g = (int)(blk % (unsigned)NG); blk /= (unsigned)NG;
  const long b = blk;
  const int Y2 = y3 - P3, X2 = x3 - P3;  // g^(2) window origin (T_3 has stride 1)
  const int Y1 = Y2 - P2, X1 = X2 - P2;  // g^(1) window origin
  const int H2 = t2.out_h, Wd2 = t2.out_w, H1 = t1.out_h, Wd1 = t1.out_w;
  const long pb = b * pstride;

  // (1) parameters of both windows
  for (int e = threadIdx.x; e < E2 + E1; e += NT) {
    float lo = 0.f, up = 0.f, bu = 0.f, z = 0.f;
    if (e < E2) {
      const int c2 = e / N2, p = e - c2 * N2;
      const int y = Y2 + p / K3, x = X2 + p % K3;
      if (y >= 0 && y < H2 && x >= 0 && x < Wd2) {
        const long ni = ((long)c2 * H2 + y) * Wd2 + x;
        lo = a_lo[pb + poff2 + ni];
        up = a_up[pb + poff2 + ni];
        bu = b_up[pb + poff2 + ni];
        z = bias[poff2 + ni];
      }
      p2s[e] = float4v{lo, up, bu, z};
    } else {
      const int f = e - E2;
      const int c1 = f / N1, p = f - c1 * N1;
      const int y = Y1 + p / W1W, x = X1 + p % W1W;
      if (y >= 0 && y < H1 && x >= 0 && x < Wd1) {
        const long ni = ((long)c1 * H1 + y) * Wd1 + x;
        lo = a_lo[pb + poff1 + ni];
        up = a_up[pb + poff1 + ni];
        bu = b_up[pb + poff1 + ni];
        z = bias[poff1 + ni];
      }
      p1s[f] = float4v{lo, up, bu, z};
    }
  }
  __syncthreads();

  // (2) relaxed g^(2) window of the 16 rows
  {
    const int row = threadIdx.x & 15, part = threadIdx.x >> 4;
    const P2Row pr = p2_row(C3, g, row);
    const float sgn = pr.neg ? -1.f : 1.f;
    const float* w3 = t3.W + (long)pr.c2 * E2;  // [C2][K3][K3] of output channel c3
    float bpart = 0.f;
    for (int e = part; e < E2; e += RP) {
      const int c2 = e / N2, p = e - c2 * N2;
      const float w = sgn * w3[e];
      const float4v q = p2s[e];
      const float v = w >= 0.f ? w * q[0] : w * q[1];
      bpart = fmaf(fminf(w, 0.f), q[2], bpart);
      bpart = fmaf(v, q[3], bpart);
      tile2[c2 * CS2 + p * 16 + row] = v;
    }
    rb2[part * 16 + row] = bpart;
  }
  __syncthreads();

  // (3) T_2^T: A over the g^(1) window, two positions per MFMA, relaxed into tile1
  {
    static_assert(C1 == 8, "the position-pair gather takes 8 channels");
    const float bpart =
        gather_pair8<C2, K2, K3, W1W, NW, false>(t2.W, tile2, CS2, tile1, CS1, p1s);
    rb1[(wave * 4 + G) * 16 + n] = bpart;
  }
  __syncthreads();

  // (4) T_1^T over the g^(1) window, one wave per input channel c0 of T_1
  {
    float l1 = wave < t1.in_c ? t1t_window_l1<W1W, K1, S1, KS1, CS1>(t1, wave, tile1,
                                                                    Y1 * S1 - P1, X1 * S1 - P1)
                              : 0.f;
    l1 += __shfl_xor(l1, 16, 64);
    l1 += __shfl_xor(l1, 32, 64);
    if (lane < 16) rl1[wave * 16 + lane] = l1;
  }
  __syncthreads();
  // (5) the bound of each row
  if (threadIdx.x >= 16) return;
  const int row = threadIdx.x;
  const P2Row pr = p2_row(C3, g, row);
  float tb = (pr.neg ? -1.f : 1.f) * t3.b[pr.c2];
  for (int q = 0; q < RP; ++q) tb += rb2[q * 16 + row];
  for (int q = 0; q < NW * 4; ++q) tb += rb1[q * 16 + row];
  float ta = 0.f;
  for (int w = 0; w < NW; ++w) ta += rl1[w * 16 + row];
  const float v = tb - eps * ta;
  const long j = ((long)pr.c2 * H3 + y3) * W3 + x3;
  if (pr.neg)
    U[b * n_relu + off3 + j] = -v;
  else
    L[b * n_relu + off3 + j] = v;
}

// Pass 4 restricted to each row's receptive field, when T_4 .. T_1 are convolutions with T_3 and
// T_2 of stride 1 (e.g. k4 s2, k3 s1, k3 s1 over 8 channels).  Row +-e_j of h^(4), j = (c4, y4, x4), carried through T_4
// is +-W_4[c4] on the K4 x K4 window of j on g^(3); the layer-3 relaxation and T_3^T spread it
// over a (K4 + K3 - 1)^2 window of g^(2), the layer-2 relaxation and T_2^T over a
// (K4 + K3 + K2 - 2)^2 window of g^(1), and the layer-1 relaxation and T_1^T over that window's
// footprint on x.  One block of 8 waves takes the 16 rows sharing a window (rows as in
// k_pass2_window, over the channels of h^(4)):
//  (1) stages the relaxation parameters of the three windows (zeros outside the maps),
//  (2) relaxes the g^(3) window (Eq. 6) with its intercept and bias terms,
//  (3) applies T_3^T, then T_2^T, as gathers on 16x16x4 MFMA (M = channels, K = (c, ky, kx)),
//      one window position per wave at a time, relaxing each result into the next LDS tile,
//  (4) applies T_1^T to the g^(1) tile with the rotating lane-group scheme (one wave per input
//      channel of T_1) and concretises (Eq. 8),
//  (5) writes l_j or u_j.  Arithmetically the dense pass minus products with zero.
template <int K4, int S4, int P4, int K3, int P3, int K2, int P2, int K1, int S1, int P1,
          int C1, int C2, int C3>
__global__ void __launch_bounds__(512)
    k_pass4_window(DLayer t1, DLayer t2, DLayer t3, DLayer t4, const float* __restrict__ a_lo,
                   const float* __restrict__ a_up, const float* __restrict__ b_up, long pstride,
                   long poff1, long poff2, long poff3, const float* __restrict__ bias, float eps,
                   float* __restrict__ L, float* __restrict__ U, long n_relu, long off4) {
  constexpr int NW = 8, NT = 64 * NW;
  constexpr int N3 = K4 * K4;               // g^(3) window positions
  constexpr int W2W = K4 - 1 + K3;          // g^(2) window width (T_3 has stride 1)
  constexpr int N2 = W2W * W2W;
  constexpr int W1W = W2W - 1 + K2;         // g^(1) window width (T_2 has stride 1)
  constexpr int N1 = W1W * W1W;
  constexpr int E3 = C3 * N3, E2 = C2 * N2, E1 = C1 * N1;
  constexpr int WO = (W1W - 1) * S1 + K1;   // footprint width on x
  constexpr int KS1 = C1 / 4;
  constexpr int PER1 = (K1 % S1 == 0) ? K1 / S1 : K1;
  constexpr int CS3 = N3 * 16 + (80 - (N3 * 16) % 64) % 64;
  constexpr int CS2 = N2 * 16 + (80 - (N2 * 16) % 64) % 64;
  constexpr int CS1 = N1 * 16 + (80 - (N1 * 16) % 64) % 64;
  constexpr int RP = NT / 16;               // threads per row in (2)
  static_assert(C1 % 4 == 0 && C1 <= 16 && C2 <= 16 && K1 <= 4 && K2 <= 4 && K3 <= 4 &&
                K4 <= 4, "geometry");
  // the g^(3) tile is dead once T_3^T has read it, so the g^(1) tile reuses its space
  __shared__ float tile31[C3 * CS3 > C1 * CS1 ? C3 * CS3 : C1 * CS1];
  float* const tile3 = tile31;
  float* const tile1 = tile31;
  __shared__ float tile2[C2 * CS2];
  __shared__ float4v p3s[E3];  // (a_lo, a_up, b_up, bias) of the g^(3) window
  __shared__ float4v p2s[E2];  // ... of the g^(2) window
  __shared__ float4v p1s[E1];  // ... of the g^(1) window (bias: W1 x0 + b1)
  __shared__ float rb3[RP * 16];      // bias terms of (2), per (part, row)
  __shared__ float rb2[NW * 4 * 16];  // bias terms of (3a), per (wave, lane group, row)
  __shared__ float rb1[NW * 4 * 16];  // bias terms of (3b)
  __shared__ float rl1[NW * 16];      // ||A_x||_1 partials of (4)

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int n = lane & 15, G = lane >> 4;
  const int H4 = t4.out_h, W4 = t4.out_w, C4 = t4.out_c;
  const int NG = p2_groups(C4);
  unsigned blk = xcd_range(blockIdx.x);  // 32-bit: the scalar divisions stay short
  const int x4 = (int)(blk % (unsigned)W4); blk /= (unsigned)W4;
  const int y4 = (int)(blk % (unsigned)H4); blk /= (unsigned)H4;
  const int g = (int)(blk % (unsigned)NG); blk /= (unsigned)NG;
  const long b = blk;
  const int Y3 = y4 * S4 - P4, X3 = x4 * S4 - P4;  // g^(3) window origin
  const int Y2 = Y3 - P3, X2 = X3 - P3;            // g^(2) window origin
  const int Y1 = Y2 - P2, X1 = X2 - P2;            // g^(1) window origin
  const int H3 = t3.out_h, Wd3 = t3.out_w, H2 = t2.out_h, Wd2 = t2.out_w;
  const int H1 = t1.out_h, Wd1 = t1.out_w;
  const long pb = b * pstride;

  // (1) parameters of the three windows
  auto stage = [&](int e, int Ww, int Y0, int X0, int Hm, int Wm, long poff) {
    const int c = e / (Ww * Ww), p = e - c * Ww * Ww;
    const int y = Y0 + p / Ww, x = X0 + p % Ww;
    float4v v = {0.f, 0.f, 0.f, 0.f};
    if (y >= 0 && y < Hm && x >= 0 && x < Wm) {
      const long ni = ((long)c * Hm + y) * Wm + x;
      v = float4v{a_lo[pb + poff + ni], a_up[pb + poff + ni], b_up[pb + poff + ni],
                  bias[poff + ni]};
    }
    return v;
  };
  for (int e = threadIdx.x; e < E3 + E2 + E1; e += NT) {
    if (e < E3) {
      const float4v v = stage(e, K4, Y3, X3, H3, Wd3, poff3);
      p3s[e] = v;
    } else if (e < E3 + E2) {
      const int f = e - E3;
      const float4v v = stage(f, W2W, Y2, X2, H2, Wd2, poff2);
      p2s[f] = v;
    } else {
      const int f = e - E3 - E2;
      const float4v v = stage(f, W1W, Y1, X1, H1, Wd1, poff1);
      p1s[f] = v;
    }
  }
  __syncthreads();

  // (2) relaxed g^(3) window of the 16 rows
  {
    const int row = threadIdx.x & 15, part = threadIdx.x >> 4;
    const P2Row pr = p2_row(C4, g, row);
    const float sgn = pr.neg ? -1.f : 1.f;
    const float* w4 = t4.W + (long)pr.c2 * E3;  // [C3][K4][K4] of output channel c4
    float bpart = 0.f;
    for (int e = part; e < E3; e += RP) {
      const int c3 = e / N3, p = e - c3 * N3;
      const float w = sgn * w4[e];
      const float4v q = p3s[e];
      const float v = w >= 0.f ? w * q[0] : w * q[1];
      bpart = fmaf(fminf(w, 0.f), q[2], bpart);
      bpart = fmaf(v, q[3], bpart);
      tile3[c3 * CS3 + p * 16 + row] = v;
    }
    rb3[part * 16 + row] = bpart;
  }
  __syncthreads();

  // (3) T_3^T, then T_2^T, as position-pair gathers (two destination positions per MFMA),
  // each result relaxed into the next tile
  static_assert(C2 == 8 && C1 == 8, "the position-pair gather takes 8 channels");
  rb2[(wave * 4 + G) * 16 + n] =
      gather_pair8<C3, K3, K4, W2W, NW, false>(t3.W, tile3, CS3, tile2, CS2, p2s);
  __syncthreads();
  rb1[(wave * 4 + G) * 16 + n] =
      gather_pair8<C2, K2, W2W, W1W, NW, true>(t2.W, tile2, CS2, tile1, CS1, p1s);
  __syncthreads();

  // (4) T_1^T over the g^(1) window, one wave per input channel c0 of T_1
  {
    float l1 = wave < t1.in_c ? t1t_window_l1<W1W, K1, S1, KS1, CS1>(t1, wave, tile1,
                                                                    Y1 * S1 - P1, X1 * S1 - P1)
                              : 0.f;
    l1 += __shfl_xor(l1, 16, 64);
    l1 += __shfl_xor(l1, 32, 64);
    if (lane < 16) rl1[wave * 16 + lane] = l1;
  }
  __syncthreads();
  // (5) the bound of each row
  if (threadIdx.x >= 16) return;
  const int row = threadIdx.x;
  const P2Row pr = p2_row(C4, g, row);
  float tb = (pr.neg ? -1.f : 1.f) * t4.b[pr.c2];
  for (int q = 0; q < RP; ++q) tb += rb3[q * 16 + row];
  for (int q = 0; q < NW * 4; ++q) tb += rb2[q * 16 + row];
  for (int q = 0; q < NW * 4; ++q) tb += rb1[q * 16 + row];
  float ta = 0.f;
  for (int w = 0; w < NW; ++w) ta += rl1[w * 16 + row];
  const float v = tb - eps * ta;
  const long j = ((long)pr.c2 * H4 + y4) * W4 + x4;
  if (pr.neg)
    U[b * n_relu + off4 + j] = -v;
  else
    L[b * n_relu + off4 + j] = v;
}

// Sum of v over the 16 lanes of each row of the wave, by DPP (row rotations by 8 and 4, then the
// quad permutations that swap lane pairs 2 and 1 apart): no LDS round trip.  Every lane ends
// with its row's total, each in its own order of additions, so one fixed lane is read.
__device__ __forceinline__ float row_sum16(float v) {
  auto dpp = [](float x, auto ctrl) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                         0, __builtin_bit_cast(int, x), decltype(ctrl)::value,
                                         0xF, 0xF, false));
  };
  v += dpp(v, std::integral_constant<int, 0x128>());  // row_ror:8
  v += dpp(v, std::integral_constant<int, 0x124>());  // row_ror:4
  v += dpp(v, std::integral_constant<int, 0x4E>());   // quad_perm(2,3,0,1): lane ^ 2
  v += dpp(v, std::integral_constant<int, 0xB1>());   // quad_perm(1,0,3,2): lane ^ 1
  return v;
}

// Reverse sweep of the receptive-field pass 2.  Layer-1 bounds do not depend on alpha, so the
// rows of pass 2 only feed d J / d alpha of the layer-1 neurons of their own window:
// sum over rows of w_r max(A~_r, 0) G_r, where A~_r = +-W_2[c2] is the row's coefficient before
// the layer-1 relaxation and G_r the layer-1 pre-activation at the row's witness
// x* = x0 + delta, delta = -eps sign(A_x) (zero outside the footprint), i.e.
// G_r = z1 + W_1 delta over the window.  Only rows with a nonzero weight contribute, and at an
// unstable-sparse layer 2 they are few, so the rows of a position are compacted: of the 2 C2
// rows +-e_(c2, y2, x2) (taken in the order (c2, sign)), the live ones are numbered in that
// order and slot s of the position takes live rows 16 s .. 16 s + 15 (slots past the last live
// row carry weight 0).  A block takes slot s of XW consecutive positions along x2 of one
// sub-domain; per window it rebuilds the relaxed patch and A_x over the footprint on MFMA,
// keeps delta in LDS, runs the layer-1 forward over the window on MFMA, reduces the 16 rows'
// contributions per window neuron and writes them to part[window][c1][pos] (windows numbered
// (b, slot, y2, x2)).  pflag[window] says whether the window has a live row; a window without
// writes nothing else, and a block whose windows have none stops after numbering them.  Row
// weights: w = g_l (sign +) or -g_u (sign -) of the row's layer-2 neuron.  (With 8 channels on
// T_1 and 8 windows per block, four waves per SIMD spill 84 bytes and are still faster than three
// without a spill: 6.8 against 7.7 ms per Base call of 20 Adam steps.)
template <int K1, int S1, int P1, int K2, int C1, int NW, int XW>
__global__ void __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(C1 >= 16 ? 3 : 4, 8)))
    k_pass2_window_grad(DLayer t1, DLayer t2, const float* __restrict__ a_lo,
                        const float* __restrict__ a_up, long pstride, float eps,
                        const float* __restrict__ gl, const float* __restrict__ gu,
                        const int8_t* __restrict__ code1, long n_relu, long off2,
                        const float* __restrict__ z1, float* __restrict__ part,
                        unsigned char* __restrict__ pflag) {
  static_assert(C1 % 4 == 0 && C1 <= 16 && K1 == 4, "unsupported geometry");
  constexpr int KS = C1 / 4;
  constexpr int NT = 64 * NW;
  constexpr int NPOS = K2 * K2;
  constexpr int NE = C1 * NPOS;                      // window entries
  constexpr int WO = (K2 - 1) * S1 + K1;
  constexpr int PER = (K1 % S1 == 0) ? K1 / S1 : K1;
  constexpr int CS = NPOS * 16 + (80 - (NPOS * 16) % 64) % 64;  // channel stride, 16 mod 64
  constexpr int NEL = C1 * CS;
  constexpr int RPT = NT / 16;                       // threads per row in the tile fills
  constexpr int NEP = (NE + RPT - 1) / RPT;          // tile entries per thread
  constexpr int NPP = (NE + NT - 1) / NT;            // staged window entries per thread
  static_assert(16 * XW <= NT, "row weights of the block's windows");
  __shared__ float tile[NEL];
  // delta / (-eps) = sign(A_x) over the footprint (0 outside the image), [c0][fy][fx][row]; a
  // byte per entry keeps the block's LDS small
  __shared__ signed char dl[NW * WO * WO * 16];
  __shared__ float wrow[XW][16];
  __shared__ unsigned short rid[XW][16];  // the slot's rows: 2 c2 + (sign -)
  __shared__ float4v prm[NE];  // a_lo, a_up, z1, unstable (1/0) of the window (0 outside)

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int n = lane & 15, G = lane >> 4;
  const int H2 = t2.out_h, W2 = t2.out_w, C2 = t2.out_c;
  const int NG = p2_groups(C2);
  const int nxc = W2 / XW;
  unsigned blk = xcd_range(blockIdx.x);  // 32-bit: the scalar divisions stay short
  const int x2c = (int)(blk % (unsigned)nxc); blk /= (unsigned)nxc;
  const int y2 = (int)(blk % (unsigned)H2); blk /= (unsigned)H2;
  const int g = (int)(blk % (unsigned)NG); blk /= (unsigned)NG;
  const long b = blk;
  const long win0 = ((b * NG + g) * H2 + y2) * W2 + (long)x2c * XW;  // first window's number
  const int Y1 = y2 * t2.stride - t2.pad;
  const int H1 = t1.out_h, Wd1 = t1.out_w;
  const long pb = b * pstride;

  // slot g of each position: one wave per position numbers the live rows by ballot
  for (int xi = wave; xi < XW; xi += NW) {
    int base = 0;
    for (int c0r = 0; c0r < 2 * C2; c0r += 64) {
      const int ci = c0r + lane, c2 = ci >> 1;
      float wgt = 0.f;
      if (ci < 2 * C2) {
        const long j = ((long)c2 * H2 + y2) * W2 + x2c * XW + xi;
        wgt = (ci & 1) ? -gu[b * n_relu + off2 + j] : gl[b * n_relu + off2 + j];
      }
      const bool live = wgt != 0.f;
      const unsigned long long m = __ballot(live);
      const int r = base + (int)__builtin_amdgcn_mbcnt_hi(
                               (unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u)) -
                    16 * g;
      if (live && r >= 0 && r < 16) {
        wrow[xi][r] = wgt;
        rid[xi][r] = (unsigned short)ci;
      }
      base += __popcll(m);
    }
    if (lane < 16 && 16 * g + lane >= base) {  // past the last live row
      wrow[xi][lane] = 0.f;
      rid[xi][lane] = 0;
    }
  }
  __syncthreads();  // wrow, rid
  {
    bool any = false;
#pragma unroll
    for (int xi = 0; xi < XW; ++xi)
#pragma unroll
      for (int r = 0; r < 16; ++r) any |= wrow[xi][r] != 0.f;
    if (threadIdx.x < XW) {
      bool live = false;
#pragma unroll
      for (int r = 0; r < 16; ++r) live |= wrow[threadIdx.x][r] != 0.f;
      pflag[win0 + threadIdx.x] = live ? 1 : 0;
    }
    if (!any) return;  // uniform: no window of the block has a live row
  }

  // this thread's entries of W_2 for the tile fills (row = tid mod 16, entries part,
  // part + RPT, ...), signed by the row; the rows differ from window to window
  const int row = threadIdx.x & 15, partid = threadIdx.x >> 4;
  float wv[NEP];
  auto wload = [&](int xi) {
    const int ci = rid[xi][row];
    const float sgn = (ci & 1) ? -1.f : 1.f;
    const float* w2 = t2.W + (long)(ci >> 1) * NE;
#pragma unroll
    for (int k = 0; k < NEP; ++k) {
      const int e = partid + k * RPT;
      wv[k] = e < NE ? sgn * w2[e] : 0.f;
    }
  };
  // tile place of the thread's entry k: entries k and k + TP lie TS channels apart at the same
  // position, so only the first TP places are held (the rest add an immediate LDS offset)
  constexpr int TP = NPOS / cgcd(RPT, NPOS), TS = TP * RPT / NPOS;
  int tbase[TP];
#pragma unroll
  for (int k = 0; k < TP; ++k) {
    const int e = partid + k * RPT;
    const int c1 = e / NPOS, pos = e - c1 * NPOS;
    tbase[k] = c1 * CS + pos * 16 + row;
  }
  auto toff = [&](int k) { return tbase[k % TP] + (k / TP) * TS * CS; };
  // T_1^T weights (step 2), one wave per input channel c0 of T_1
  const int c0 = wave;
  const bool cok = c0 < t1.in_c;
  float wreg[PER][KS];
  {
    const int M = lane & 15, slot = M >> 2, kx = M & 3;
#pragma unroll
    for (int ph = 0; ph < PER; ++ph) {
      const int ky = ((slot - ph * S1) % K1 + K1) % K1;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int c1 = 4 * ks + G;
        wreg[ph][ks] = (cok && slot < K1 && kx < K1)
                           ? t1.W[(((long)c1 * t1.in_c + c0) * K1 + ky) * K1 + kx] : 0.f;
      }
    }
  }
  // W_1 weights (step 3): M = 16 channels c1, one K step per (input channel, tap row) with the
  // tap column as the lane group
  static_assert(K1 == 4, "tap columns are the four lane groups");
  constexpr int NK1 = NW * K1;  // K steps: in_c == NW
  float w1r[NK1];
#pragma unroll
  for (int ks = 0; ks < NK1; ++ks) {
    const int cc = ks / K1, ky = ks % K1, c1A = lane & 15;
    w1r[ks] = (c1A < C1 && cc < t1.in_c)
                  ? t1.W[(((long)c1A * t1.in_c + cc) * K1 + ky) * K1 + G] : 0.f;
  }
  const int Hi = t1.in_h, Wi = t1.in_w;
  const int OY = Y1 * S1 - P1;

  // relaxation of a window, one entry per (thread, k), fetched a window ahead
  float4v pn[NPP];
  auto pfetch = [&](int X1) {
#pragma unroll
    for (int k = 0; k < NPP; ++k) {
      const int e = threadIdx.x + k * NT;
      pn[k] = float4v{0.f, 0.f, 0.f, 0.f};
      if (e >= NE) continue;
      const int c1 = e / NPOS, pos = e - c1 * NPOS;
      const int ky2 = pos / K2, kx2 = pos - ky2 * K2;
      const int y1 = Y1 + ky2, x1 = X1 + kx2;
      if (y1 >= 0 && y1 < H1 && x1 >= 0 && x1 < Wd1) {
        const long ni = ((long)c1 * H1 + y1) * Wd1 + x1;
        pn[k] = float4v{a_lo[pb + ni], a_up[pb + ni], z1[ni],
                        code1[b * n_relu + ni] == 5 ? 1.f : 0.f};
      }
    }
  };
  pfetch(x2c * XW * t2.stride - t2.pad);

  for (int xi = 0; xi < XW; ++xi) {
    const int x2 = x2c * XW + xi;
    const int X1 = x2 * t2.stride - t2.pad;
    float* out = part + (win0 + xi) * (long)NE;
    bool active = false;
#pragma unroll
    for (int r = 0; r < 16; ++r) active |= wrow[xi][r] != 0.f;
    if (!active) {  // uniform: no row of this window carries weight (its flag says so)
      if (xi + 1 < XW) pfetch(X1 + t2.stride);
      continue;
    }
    // (1) stage the window's relaxation; fetch the next window's; relaxed window coefficients
    wload(xi);
#pragma unroll
    for (int k = 0; k < NPP; ++k) {
      const int e = threadIdx.x + k * NT;
      if (e < NE) prm[e] = pn[k];
    }
    __syncthreads();
    if (xi + 1 < XW) pfetch(X1 + t2.stride);
#pragma unroll
    for (int k = 0; k < NEP; ++k) {
      const int e = partid + k * RPT;
      if (k + 1 < NEP || e < NE) {  // (only the last k can fall past NE)
        const float4v pr = prm[e];
        tile[toff(k)] = wv[k] * (wv[k] >= 0.f ? pr[0] : pr[1]);
      }
    }
    __syncthreads();

    // (2) A_x over the footprint; delta = -eps sign(A_x) into LDS (0 outside the image)
    const int OX = X1 * S1 - P1;
    {
      float acc[WO];
#pragma unroll
      for (int x = 0; x < WO; ++x) acc[x] = 0.f;
      auto emit = [&](int yl) {
        if (!cok) return;
        const int y = OY + yl;
#pragma unroll
        for (int x = 0; x < WO; ++x) {
          const int xc = OX + x;
          const bool in = y >= 0 && y < Hi && xc >= 0 && xc < Wi;
          const int sv = acc[x] > 0.f ? 1 : (acc[x] < 0.f ? -1 : 0);
          dl[((c0 * WO + yl) * WO + x) * 16 + n] = (signed char)(in ? sv : 0);
        }
      };
#pragma unroll
      for (int j = 0; j < K2; ++j) {
        const int ph = j % PER;
#pragma unroll
        for (int i = 0; i < K2; ++i) {
          const int pos = j * K2 + i;
          float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ph][ks],
                                                    tile[(4 * ks + G) * CS + pos * 16 + n],
                                                    d, 0, 0, 0);
#pragma unroll
          for (int kx2 = 0; kx2 < K1; ++kx2) acc[i * S1 + kx2] += d[kx2];
        }
        const int ky = ((G - ph * S1) % K1 + K1) % K1;
        if (G < K1 && ky < S1) {
          emit(j * S1 + ky);
#pragma unroll
          for (int x = 0; x < WO; ++x) acc[x] = 0.f;
        }
      }
      {
        const int ky = ((G - ((K2 - 1) % PER) * S1) % K1 + K1) % K1;
        if (G < K1 && ky >= S1) emit((K2 - 1) * S1 + ky);
      }
    }
    __syncthreads();

    // the tile now holds max(A~, 0), the non-negative parts of the unrelaxed window coefficients
#pragma unroll
    for (int k = 0; k < NEP; ++k) {
      const int e = partid + k * RPT;
      if (k + 1 < NEP || e < NE) tile[toff(k)] = fmaxf(wv[k], 0.f);
    }
    __syncthreads();

    // (3) G = z1 + W_1 delta = z1 - eps W_1 sign(A_x) at each window neuron, W_1 sign(A_x) on
    // MFMA (the footprint entry of a K step is uniform per lane group); contributions summed
    // over the rows
    {
      const float wn = wrow[xi][n];
      for (int pos = wave; pos < NPOS; pos += NW) {
        const int j = pos / K2, i = pos - j * K2;
        float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NK1; ++ks) {
          const int cc = ks / K1, ky = ks % K1;
          const float bv = (float)dl[((cc * WO + j * S1 + ky) * WO + i * S1 + G) * 16 + n];
          d = __builtin_amdgcn_mfma_f32_16x16x4f32(w1r[ks], bv, d, 0, 0, 0);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int c1 = 4 * G + r;
          float cval = 0.f;
          if (c1 < C1) {
            const int e = c1 * NPOS + pos;
            const float4v pr = prm[e];
            cval = wn * pr[3] * tile[c1 * CS + pos * 16 + n] * fmaf(-eps, d[r], pr[2]);
          }
          cval = row_sum16(cval);
          if (n == 0 && c1 < C1) out[c1 * NPOS + pos] = cval;
        }
      }
    }
    __syncthreads();  // prm, tile and dl are refilled by the next window
  }
}

// The sum for neuron ni = (c1, y1, x1) of sub-domain b: the flagged partials of the windows that
// cover it, in the order (g, ky2, kx2), which the neuron alone fixes.
__device__ __forceinline__ float p2_gather_neuron(long b, long ni, const DLayer& t1,
                                                  const DLayer& t2, int NPOS,
                                                  const float* __restrict__ part,
                                                  const unsigned char* __restrict__ pflag) {
  const int hw = t1.out_h * t1.out_w;
  const int c1 = (int)(ni / hw), y1 = (int)((ni / t1.out_w) % t1.out_h), x1 = (int)(ni % t1.out_w);
  const int H2 = t2.out_h, W2 = t2.out_w, K2 = t2.k, S2 = t2.stride, P2 = t2.pad;
  const int NG = p2_groups(t2.out_c);
  const int C1 = t1.out_c;
  // the windows covering (y1, x1): taps ky2 = (y1 + P2) mod S2, + S2, ... (the same for x)
  const int ry = (y1 + P2) % S2, rx = (x1 + P2) % S2;
  float acc = 0.f;
  for (int g = 0; g < NG; ++g)
    for (int ky2 = ry; ky2 < K2; ky2 += S2) {
      const int yn = y1 + P2 - ky2;
      if (yn < 0) break;  // (yn falls as ky2 grows)
      const int y2 = yn / S2;
      if (y2 >= H2) continue;
      for (int kx2 = rx; kx2 < K2; kx2 += S2) {
        const int xn = x1 + P2 - kx2;
        if (xn < 0) break;
        const int x2 = xn / S2;
        if (x2 >= W2) continue;
        const long blk = ((b * NG + g) * H2 + y2) * W2 + x2;
        if (pflag[blk]) acc += part[(blk * C1 + c1) * NPOS + ky2 * K2 + kx2];
      }
    }
  return acc;
}

// d J / d alpha of layer-1 neuron (c1, y1, x1) from pass 2: the partial sums of every window that
// covers the neuron, in a fixed order; a thread per (sub-domain, neuron).
__global__ void __launch_bounds__(kBlock)
    k_pass2_grad_gather(long nb, DLayer t1, DLayer t2, int NPOS, const float* __restrict__ part,
                        const unsigned char* __restrict__ pflag,
                        const int8_t* __restrict__ code1, long n_relu,
                        float* __restrict__ ga1) {
  long idx = blockIdx.x * (long)blockDim.x + threadIdx.x;
  const long n1 = (long)t1.out_c * t1.out_h * t1.out_w;
  if (idx >= nb * n1) return;
  const long b = idx / n1, ni = idx % n1;
  if (code1[b * n_relu + ni] != 5) return;
  ga1[b * n_relu + ni] += p2_gather_neuron(b, ni, t1, t2, NPOS, part, pflag);
}

// The same over the sub-domain's unstable layer-1 neurons listed by k_unstable_index
// (list[b][k], cnt[b]): a block per sub-domain, a thread per listed neuron, the same sums.
__global__ void __launch_bounds__(kBlock)
    k_pass2_grad_gather_c(DLayer t1, DLayer t2, int NPOS, const float* __restrict__ part,
                          const unsigned char* __restrict__ pflag, const int* __restrict__ list,
                          const int* __restrict__ cnt, long n1, long n_relu,
                          float* __restrict__ ga1) {
  const long b = blockIdx.x;
  const int m = cnt[b];
  for (int k = threadIdx.x; k < m; k += blockDim.x) {
    const long ni = list[b * n1 + k];
    ga1[b * n_relu + ni] += p2_gather_neuron(b, ni, t1, t2, NPOS, part, pflag);
  }
}

// Linear^T as a GEMM on 32x32x2 MFMA: out[i][q] = sum_o W[o][i] in[o][q].  Block: 32 rows q
// and 8 waves; the block's inputs in[.][q0..q0+31] sit in LDS, each wave takes every 8th tile of
// 32 output features i, K runs over o two at a time with the A operand (W, read straight from
// memory, L2-resident) fetched one group of 16 steps ahead.  Epilogue as in the other stages.
template <int MODE, int NWAVE>
__global__ void __launch_bounds__(64 * NWAVE) k_fcT_mfma(DLayer t, const float* __restrict__ in,
                                                  long ldq, long Q, Sink s) {
  extern __shared__ float lds[];
  float* tile = lds;                            // [out_c][32]
  float* red = lds + (long)t.out_c * 32;        // [NWAVE][3][32]
  const int lane = threadIdx.x & 63, wave = wave_id(), nw = blockDim.x >> 6;
  const int n = lane & 31, h = lane >> 5;
  const long q0 = (long)blockIdx.x * 32;
  const long q = q0 + n;
  const long b = q < Q ? q / s.R : 0;
  const int nin = t.in_c, nout = t.out_c;
  for (int e = threadIdx.x; e < nout * 8; e += blockDim.x) {
    const int j4 = e & 7, o = e >> 3;
    *reinterpret_cast<float4v*>(tile + o * 32 + j4 * 4) =
        *reinterpret_cast<const float4v*>(in + (long)o * ldq + q0 + j4 * 4);
  }
  __syncthreads();
  Acc sum{0.f, 0.f, 0.f};
  const int KS = (nout + 1) / 2;
  constexpr int U = NWAVE > 8 ? 8 : 16;
  for (int mt = wave; mt * 32 < nin; mt += nw) {
    floatx16 d;
#pragma unroll
    for (int r = 0; r < 16; ++r) d[r] = 0.f;
    const int ia = mt * 32 + (lane & 31);
    const bool iok = ia < nin;
    float an[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int o = 2 * u + h;
      an[u] = (o < nout && iok) ? t.W[(long)o * nin + ia] : 0.f;
    }
    for (int k0 = 0; k0 < KS; k0 += U) {
      float a[U];
#pragma unroll
      for (int u = 0; u < U; ++u) a[u] = an[u];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int o = 2 * (k0 + U + u) + h;
        an[u] = (o < nout && iok) ? t.W[(long)o * nin + ia] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int o = 2 * (k0 + u) + h;
        const float bv = o < nout ? tile[o * 32 + n] : 0.f;
        d = __builtin_amdgcn_mfma_f32_32x32x2f32(a[u], bv, d, 0, 0, 0);
      }
    }
    if (q < Q) {
      // accumulator r holds feature i = mt*32 + 8 (r/4) + 4h + r%4: four runs of four
      // consecutive features.  Every operand of the epilogue is loaded before the first store
      // (the stores could alias them as far as the compiler knows, so it would not hoist them).
      auto ld4 = [&](const float* p, int i0) {
        if (i0 + 4 <= nin) return *reinterpret_cast<const float4v*>(p + i0);
        float4v v = {0.f, 0.f, 0.f, 0.f};
        for (int e = 0; e < 4; ++e)
          if (i0 + e < nin) v[e] = p[i0 + e];
        return v;
      };
      float4v p0[4], p1[4], p2[4], p3[4];
      const long pb = b * s.pstride;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int i0 = mt * 32 + 8 * g + 4 * h;
        if constexpr (MODE == MODE_SLAB) {
          p0[g] = ld4(s.a_lo + pb, i0);
          p1[g] = ld4(s.a_up + pb, i0);
          p2[g] = ld4(s.b_up + pb, i0);
          p3[g] = ld4(s.bias, i0);  // per-neuron bias vector (bias_hw == 1)
        } else {
          p0[g] = s.x0 ? ld4(s.x0, i0) : float4v{0.f, 0.f, 0.f, 0.f};
        }
      }
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = mt * 32 + 8 * g + 4 * h + e;
          if (i >= nin) continue;
          const float a = d[4 * g + e];
          if constexpr (MODE == MODE_SLAB) {
            if (s.tape) s.tape[(long)i * s.ldq + q] = a;
          } else {
            if (s.tsign) s.tsign[(long)i * s.ldq + q] = sign8(a);
          }
          if constexpr (MODE == MODE_SLAB) {
            const float ah = a * (a >= 0.f ? p0[g][e] : p1[g][e]);
            sum.beta = fmaf(fminf(a, 0.f), p2[g][e], sum.beta);
            sum.beta = fmaf(ah, p3[g][e], sum.beta);
            s.out[(long)i * s.ldq + q] = ah;
          } else {
            sum.lin = fmaf(a, p0[g][e], sum.lin);
            sum.l1 += fabsf(a);
          }
        }
    }
  }
  block_finish<MODE>(s, sum, red, q0, Q, false);
}

// The final pass's first two stages when T_L and T_{L-1} are fully connected, 16 rows
// q = (b, s) per block (NW waves):
//  (1) row q is the spec row C_s over h^(L) (the property merged into the last layer, Sec. 2.1);
//      through T_L it becomes C_s W_L over g^(L-1) with bias C_s b_L (Eq. 4), both formed once
//      per call by k_setup (wsp).  Its entries are relaxed onto layer L-1 (Eq. 6) into an LDS
//      tile [j][16 q] with their intercept and bias terms;
//  (2) T_{L-1}^T on 16x16x4 MFMA (M = 16 features i of g^(L-2), K = 4 features j, N = 16 rows),
//      one 16-feature tile per wave at a time with its operands from W_{L-1} (L2-resident); the
//      results are relaxed onto layer L-2 and stored into the slab, with their terms.
// The rows' bias goes to Sink::beta (the pass's first stage).  lo1/up1/bu1/bias1: the
// relaxation of layer L-1; s: that of layer L-2 and the slab.
// NK = ceil(n_{L-1} / 4) k-steps.
template <int NW, int NK>
__global__ void __launch_bounds__(64 * NW)
    k_final_fc(DLayer tM, const float* __restrict__ wsp, int S, long nb, long Q,
               const float* __restrict__ lo1, const float* __restrict__ up1,
               const float* __restrict__ bu1, const float* __restrict__ bias1, Sink s) {
  extern __shared__ float lds[];
  const int nj = tM.out_c, ni = tM.in_c;  // n_{L-1}, n_{L-2}
  const int KP = (nj + 3) & ~3;
  float* tile = lds;                 // [KP][16]
  float* red = lds + KP * 16;        // [NW * 64] terms of (1), then [NW][16] terms of (2)
  const int lane = threadIdx.x & 63, wave = wave_id();
  const long q0 = (long)blockIdx.x * 16;
  // (1) thread: row qa = tid & 15, features j = tid >> 4 + k NW 4
  {
    const int qa = threadIdx.x & 15;
    const long q = min(q0 + qa, Q - 1);
    const long b = q / S;
    const int sr = (int)(q % S);
    const long pb = b * s.pstride;
    float beta = 0.f;
    for (int j = threadIdx.x >> 4; j < KP; j += NW * 4) {
      float ah = 0.f;
      if (j < nj) {
        const float a = wsp[(long)sr * nj + j];
        ah = a * (a >= 0.f ? lo1[pb + j] : up1[pb + j]);
        beta = fmaf(fminf(a, 0.f), bu1[pb + j], beta);
        beta = fmaf(ah, bias1[j], beta);
      }
      tile[j * 16 + qa] = ah;
    }
    red[threadIdx.x] = beta;
  }
  __syncthreads();
  // (2) A tile's operands are loaded at once: the column of W_{L-1} (one entry per k-step;
  // entries j >= n_{L-1} read a clamped row and meet zeros of the LDS tile) and the four
  // neurons' relaxation as float4.
  const int n = lane & 15, G = lane >> 4;
  const long q = q0 + n;
  const long b = (q < Q ? q : Q - 1) / S;
  const long pb = b * s.pstride;
  float beta = 0.f;
  struct Ops {
    float a[NK];
    float4v lo, up, bu, bz;
  };
  auto load = [&](int mt, Ops& o) {
    const int ia = min(mt * 16 + n, ni - 1);
    const float* w = tM.W + (long)G * ni + ia;
    // 4 k + G < 4 (NK - 1) < n_{L-1} for k < NK - 1
#pragma unroll
    for (int k = 0; k < NK - 1; ++k) o.a[k] = w[(long)4 * k * ni];
    o.a[NK - 1] = tM.W[(long)min(4 * (NK - 1) + G, nj - 1) * ni + ia];
    // within the padded segment round_up(ni, 4); a clamped quad has no neuron i < ni
    const long i0 = min(mt * 16 + 4 * G, ((ni + 3) & ~3) - 4);
    o.lo = *reinterpret_cast<const float4v*>(s.a_lo + pb + i0);
    o.up = *reinterpret_cast<const float4v*>(s.a_up + pb + i0);
    o.bu = *reinterpret_cast<const float4v*>(s.b_up + pb + i0);
    o.bz = *reinterpret_cast<const float4v*>(s.bias + i0);
  };
  auto compute = [&](int mt, const Ops& o) {
    float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < NK; ++k)
      d = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a[k], tile[(4 * k + G) * 16 + n], d, 0, 0, 0);
    // lane holds features i0 .. i0 + 3 of row q
    const int i0 = mt * 16 + 4 * G;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + r;
      if (i < ni) {
        const float a = d[r];
        const float ah = a * (a >= 0.f ? o.lo[r] : o.up[r]);
        beta = fmaf(fminf(a, 0.f), o.bu[r], beta);
        beta = fmaf(ah, o.bz[r], beta);
        s.out[(long)i * s.ldq + q] = ah;
      }
    }
  };
  const int ntile = (ni + 15) / 16;
  for (int mt = wave; mt < ntile; mt += NW) {
    Ops o;
    load(mt, o);
    compute(mt, o);
  }
  // (2)'s terms per row: over the lane groups, then over the waves in order; (1)'s: over the
  // threads of the row in order
  beta += __shfl_xor(beta, 16, 64);
  beta += __shfl_xor(beta, 32, 64);
  if (lane < 16) red[NW * 64 + wave * 16 + lane] = beta;
  __syncthreads();
  if (threadIdx.x < 16) {
    const long qq = q0 + threadIdx.x;
    if (qq < Q) {
      float tb = wsp[(long)S * nj + qq % S];
      for (int t = threadIdx.x; t < NW * 64; t += 16) tb += red[t];
      for (int w = 0; w < NW; ++w) tb += red[NW * 64 + w * 16 + threadIdx.x];
      s.beta[qq] = tb;
    }
  }
}

// Relaxation parameters of ReLU layer m for every sub-domain of the chunk (Eq. 5 with the split
// override of Sec. 3.1, checked in the order: split, u <= 0, l >= 0, unstable).
// lsh, ush (optional): bounds shared by every sub-domain (layer 1), copied into its rows of l, u.
__global__ void __launch_bounds__(kBlock)
    k_relax_params(long nb, long nm, long stride, long off, long pstride, long poff,
                   float* __restrict__ l, float* __restrict__ u,
                   const float* __restrict__ lsh, const float* __restrict__ ush,
                   const int8_t* __restrict__ split, const float* __restrict__ alpha,
                   float* __restrict__ a_lo, float* __restrict__ a_up, float* __restrict__ b_up,
                   int8_t* __restrict__ code, const float* __restrict__ lpar,
                   const float* __restrict__ upar) {
  long idx = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (idx >= nb * nm) return;
  long b = idx / nm, j = idx % nm;
  long p = b * stride + off + j;
  long pp = b * pstride + poff + j;
  const int sp = split ? split[p] : 0;
  float lj = lsh ? lsh[j] : l[p], uj = ush ? ush[j] : u[p];
  parent_clip(lj, uj, lpar, upar, p);
  if (lsh || lpar) {
    l[p] = lj;
    u[p] = uj;
  }
  const Relax1 r = relax_neuron(lj, uj, sp, alpha ? alpha + p : nullptr);
  a_lo[pp] = r.lo;
  a_up[pp] = r.up;
  b_up[pp] = r.bu;
  code[p] = (int8_t)r.code;
}

// The same with four consecutive neurons per thread (float4 and 32-bit accesses), when the
// layer's segments and every array are 4-aligned (checked by the caller).
__global__ void __launch_bounds__(kBlock)
    k_relax_params4(long nb, long nm4, long stride, long off, long pstride, long poff,
                    float* __restrict__ l, float* __restrict__ u,
                    const float* __restrict__ lsh, const float* __restrict__ ush,
                    const int8_t* __restrict__ split, const float* __restrict__ alpha,
                    float* __restrict__ a_lo, float* __restrict__ a_up, float* __restrict__ b_up,
                    int8_t* __restrict__ code, const float* __restrict__ lpar,
                    const float* __restrict__ upar) {
  long idx = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (idx >= nb * nm4) return;
  long b = idx / nm4, j = (idx % nm4) * 4;
  long p = b * stride + off + j;
  long pp = b * pstride + poff + j;
  float4v lv, uv;
  if (lsh) {
    lv = *reinterpret_cast<const float4v*>(lsh + j);
    uv = *reinterpret_cast<const float4v*>(ush + j);
  } else {
    lv = *reinterpret_cast<const float4v*>(l + p);
    uv = *reinterpret_cast<const float4v*>(u + p);
  }
  if (lpar) {
    const float4v pl = *reinterpret_cast<const float4v*>(lpar + p);
    const float4v pu = *reinterpret_cast<const float4v*>(upar + p);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      lv[r] = fmaxf(lv[r], pl[r]);
      uv[r] = fminf(uv[r], pu[r]);
    }
  }
  if (lsh || lpar) {
    *reinterpret_cast<float4v*>(l + p) = lv;
    *reinterpret_cast<float4v*>(u + p) = uv;
  }
  const int sp4 = split ? *reinterpret_cast<const int*>(split + p) : 0;
  float4v lo, up, bu;
  int cd = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const Relax1 rx = relax_neuron(lv[r], uv[r], (int)(int8_t)(sp4 >> (8 * r)),
                                   alpha ? alpha + p + r : nullptr);
    lo[r] = rx.lo;
    up[r] = rx.up;
    bu[r] = rx.bu;
    cd |= (rx.code & 0xff) << (8 * r);
  }
  *reinterpret_cast<float4v*>(a_lo + pp) = lo;
  *reinterpret_cast<float4v*>(a_up + pp) = up;
  *reinterpret_cast<float4v*>(b_up + pp) = bu;
  *reinterpret_cast<int*>(code + p) = cd;
}

// ---------------------------------------------------------------------------------------------
// Gradient kernels (reverse sweep of one pass)
// ---------------------------------------------------------------------------------------------

// Row weights of pass P: 1 for the spec rows of the final pass (J = sum_s lb_s); for pass P < L
// the adjoints of the bounds it produced: row +e_j carries g_l[j], row -e_j carries -g_u[j]
// (u_j = -lb of that row); the two signs in halves of R, or interleaved (inter).
__global__ void __launch_bounds__(kBlock) k_row_weights(long Q, long R, long nP, long n_relu,
                                                        long offP, int final_pass, int inter,
                                                        const float* __restrict__ gl,
                                                        const float* __restrict__ gu,
                                                        float* __restrict__ w) {
  long q = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (q >= Q) return;
  if (final_pass) {
    w[q] = 1.f;
    return;
  }
  long b = q / R, r = q % R;
  if (inter)  // rows 2j, 2j + 1: +e_j, -e_j
    w[q] = (r & 1) ? -gu[b * n_relu + offP + (r >> 1)] : gl[b * n_relu + offP + (r >> 1)];
  else
    w[q] = r < nP ? gl[b * n_relu + offP + r] : -gu[b * n_relu + offP + (r - nP)];
}

// Forward step of the witness pass through layer m for every row with a non-zero weight.
// The row's bound equals its linear lower function at the box vertex x* = x0 - eps sign(A_x);
// that function is the network with each ReLU replaced, per row, by the line the backward pass
// chose for it (lower line where the row's coefficient was >= 0, upper line otherwise).
// G = W_m z + b_m is the pre-activation along that network; z_out = chosen line applied to G.
// WITNESS: the input z is built on the fly from the sign tape of A_x; the input pointer then
// holds one int8_t sign per entry, [i][ldq].
//
// On 16x16x4 MFMA, for conv and linear layers alike (a linear layer is a 1x1 convolution on a
// 1x1 map): implicit GEMM with M = 16 output channels co, N = 16 rows q
// and K = (ci, ky, kx), four per instruction.  Block: 16 rows x 4 waves; output positions are
// dealt round-robin to the waves.  A block whose 16 rows all carry weight 0 exits at once.
template <bool WITNESS>
__global__ void __launch_bounds__(256)
    k_fwd_mfma(DLayer t, const float* __restrict__ zin, unsigned ldq, unsigned Q, long R,
               const float* __restrict__ w, const float* __restrict__ x0, float eps,
               const float* __restrict__ tape, const float* __restrict__ a_lo,
               const float* __restrict__ a_up, const float* __restrict__ b_up, long pstride,
               float* __restrict__ G, float* __restrict__ zout) {
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int n = lane & 15, g = lane >> 4;
  const unsigned q0 = xcd_tile(blockIdx.x) * 16u;
  if (q0 >= Q) return;  // grid padding, uniform per block
  const unsigned q = q0 + n;
  const bool qok = q < Q;
  const float wq = qok ? w[q] : 0.f;
  if (__syncthreads_or(wq != 0.f) == 0) return;  // uniform: the whole block is idle
  const unsigned b = qok ? q / (unsigned)R : 0u;
  const int K = t.k > 0 ? t.k : 1;
  const int KD = t.in_c * K * K;
  const int nks = (KD + 3) / 4;
  const int Hout = t.out_h, Wout = t.out_w, Hin = t.in_h, Win = t.in_w;
  const int npos = Hout * Wout;
  const int nmt = (t.out_c + 15) / 16;
  // work items (output position, 16-channel M tile) dealt to the 4 waves, so that a layer with
  // one position (Linear) keeps every wave busy; the operands of 8 K steps are loaded at once
  for (int it = wave; it < npos * nmt; it += 4) {
    const int pos = it / nmt, mt = it - pos * nmt;
    const int y = pos / Wout, x = pos - y * Wout;
    const int yb = y * t.stride - t.pad, xb = x * t.stride - t.pad;
    {
      const int coA = mt * 16 + n;  // A operand row (M = l%16)
      auto operands = [&](int ks, float& av, float& bv) {
        const int kk = ks * 4 + g;  // K index of this lane group
        av = 0.f;
        bv = 0.f;
        if (kk < KD) {
          const int ci = kk / (K * K), rem = kk - ci * K * K;
          const int ky = rem / K, kx = rem - ky * K;
          if (coA < t.out_c) av = t.W[(long)coA * KD + kk];
          const int yi = yb + ky, xi = xb + kx;
          if (yi >= 0 && yi < Hin && xi >= 0 && xi < Win) {
            const unsigned ii = ((unsigned)ci * Hin + yi) * Win + xi;
            if constexpr (WITNESS)
              bv = x0[ii] - eps * (float)reinterpret_cast<const int8_t*>(zin)[(size_t)ii * ldq + q];
            else
              bv = zin[ii * ldq + q];
          }
        }
      };
      float4v d = {0.f, 0.f, 0.f, 0.f};
      int ks = 0;
      for (; ks + 8 <= nks; ks += 8) {
        float av[8], bv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) operands(ks + u, av[u], bv[u]);
#pragma unroll
        for (int u = 0; u < 8; ++u) d = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], bv[u], d, 0, 0, 0);
      }
      for (; ks < nks; ++ks) {
        float av, bv;
        operands(ks, av, bv);
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, d, 0, 0, 0);
      }
      if (!qok || wq == 0.f) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = mt * 16 + 4 * g + r;
        if (co >= t.out_c) continue;
        const float gv = d[r] + t.b[co];
        const unsigned o = ((unsigned)co * Hout + y) * Wout + x;
        const unsigned idx = o * ldq + q;
        G[idx] = gv;
        if (zout) {
          const long pi = (long)b * pstride + o;
          zout[idx] = tape[idx] >= 0.f ? a_lo[pi] * gv : fmaf(a_up[pi], gv, b_up[pi]);
        }
      }
    }
  }
}

// The witness forward step through a Linear layer past the first (its input z is a
// [in][ldq] slab), as a GEMM on 16x16x4 MFMA: M = 16 outputs o, N = 16 rows q, K = inputs.
// Block: 64 rows (one N tile per wave) and every output (MT tiles of 16 per wave).  K runs in
// chunks of 32 staged in LDS, the inputs as [k][q] and the weights as [o][k], double-buffered:
// the next chunk's global loads are issued before the current chunk's MFMAs and parked after
// them.  Epilogue as in k_fwd_mfma; rows without weight (and rows past Q, which read the
// slab's padding) are computed but never stored.  in_c is a multiple of 4.
template <int MT>
__global__ void __launch_bounds__(256)
    k_fwd_fc(DLayer t, const float* __restrict__ zin, unsigned ldq, unsigned Q, long R,
             const float* __restrict__ w, const float* __restrict__ tape,
             const float* __restrict__ a_lo, const float* __restrict__ a_up,
             const float* __restrict__ b_up, long pstride, float* __restrict__ G,
             float* __restrict__ zout) {
  constexpr int KC = 32;
  constexpr int ZS = 80;       // row stride of the input chunk: the 4 lane groups' reads of a
                               // K step fall on distinct banks
  constexpr int WS = KC + 4;   // row stride of the weight chunk (likewise for the 16 outputs)
  constexpr int NW4 = MT * 16 * KC / 4;         // float4 of a weight chunk
  constexpr int WPT = (NW4 + 255) / 256;
  __shared__ __attribute__((aligned(16))) float zs[2][KC * ZS];
  __shared__ __attribute__((aligned(16))) float ws[2][MT * 16 * WS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 15, g = lane >> 4;
  const unsigned q0 = xcd_range(blockIdx.x) * 64u;
  if (q0 >= Q) return;  // grid padding, uniform per block
  const unsigned q = q0 + 16u * wave + n;
  const float wq = q < Q ? w[q] : 0.f;
  if (__syncthreads_or(wq != 0.f) == 0) return;  // uniform: the whole block is idle
  const int nin = t.in_c, nout = t.out_c;
  const int nch = (nin + KC - 1) / KC;
  float4v zr[2], wr[WPT];
  auto fetch = [&](int c) {
    const int k0 = c * KC;
#pragma unroll
    for (int k = 0; k < 2; ++k) {  // inputs: 32 x 64 floats, float4 e = (k, quarter of 16 rows)
      const int e = tid + 256 * k, kk = e >> 4, q4 = e & 15;
      zr[k] = k0 + kk < nin
                  ? *reinterpret_cast<const float4v*>(zin + (size_t)(k0 + kk) * ldq + q0 + 4 * q4)
                  : float4v{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int k = 0; k < WPT; ++k) {  // weights: MT 16 x 32 floats, float4 e = (o, k quarter)
      const int e = tid + 256 * k, o = e >> 3, k4 = e & 7;
      wr[k] = (e < NW4 && o < nout && k0 + 4 * k4 < nin)
                  ? *reinterpret_cast<const float4v*>(t.W + (size_t)o * nin + k0 + 4 * k4)
                  : float4v{0.f, 0.f, 0.f, 0.f};
    }
  };
  auto park = [&](int buf) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int e = tid + 256 * k, kk = e >> 4, q4 = e & 15;
      *reinterpret_cast<float4v*>(&zs[buf][kk * ZS + 4 * q4]) = zr[k];
    }
#pragma unroll
    for (int k = 0; k < WPT; ++k) {
      const int e = tid + 256 * k, o = e >> 3, k4 = e & 7;
      if (e < NW4) *reinterpret_cast<float4v*>(&ws[buf][o * WS + 4 * k4]) = wr[k];
    }
  };
  float4v d[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) d[mt] = float4v{0.f, 0.f, 0.f, 0.f};
  fetch(0);
  park(0);
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    const int buf = c & 1;
    if (c + 1 < nch) fetch(c + 1);
#pragma unroll
    for (int ks = 0; ks < KC / 4; ++ks) {
      const float bv = zs[buf][(4 * ks + g) * ZS + 16 * wave + n];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        d[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(ws[buf][(mt * 16 + n) * WS + 4 * ks + g], bv,
                                                     d[mt], 0, 0, 0);
    }
    if (c + 1 < nch) park(buf ^ 1);
    __syncthreads();
  }
  // lane (n, g) holds outputs mt 16 + 4 g + r of row q
  if (q >= Q || wq == 0.f) return;
  const long b = q / R;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int o = mt * 16 + 4 * g + r;
      if (o >= nout) continue;
      const float gv = d[mt][r] + t.b[o];
      const size_t idx = (size_t)o * ldq + q;
      G[idx] = gv;
      if (zout) {  // both lines, then a select (no branch around the loads)
        const long pi = b * pstride + o;
        const float zl = a_lo[pi] * gv, zu = fmaf(a_up[pi], gv, b_up[pi]);
        zout[idx] = tape[idx] >= 0.f ? zl : zu;
      }
    }
}

// Sum over each group of 8 consecutive lanes (lanes 8k..8k+7), valid in lanes 8k..8k+3: two
// butterfly steps inside each quad, then the quad 4 lanes up (DPP, no LDS; a row rotation by r
// hands lane i the value of lane i - r of its row of 16).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float sum8(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm(1,0,3,2): lane ^ 1
  v += dpp_f<0x4E>(v);   // quad_perm(2,3,0,1): lane ^ 2
  v += dpp_f<0x12C>(v);  // row_ror:12: lane i reads lane (i + 4) mod 16 of its row
  return v;
}

// A copy of a k x k convolution's weights with the two tap indices exchanged,
// Wt[co][ci][kx][ky] = W[co][ci][ky][kx], so that the taps of one column are contiguous.
__global__ void __launch_bounds__(kBlock)
    k_taps_swap(long n, int k, const float* __restrict__ W, float* __restrict__ Wt) {
  const long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i >= n) return;
  const long kk = (long)k * k, base = i / kk * kk;
  const int ky = (int)(i % kk) / k, kx = (int)(i % k);
  Wt[base + (long)kx * k + ky] = W[i];
}

// A copy of a Linear layer's weights over a C x HW input with the input index reordered
// channel-last: Wc[j][p C + c] = W[j][c HW + p], so that the entries of one input position
// over all channels are contiguous.
__global__ void __launch_bounds__(kBlock)
    k_fc_chlast(long n, int C, int HW, const float* __restrict__ W, float* __restrict__ Wc) {
  const long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i >= n) return;
  const long nin = (long)C * HW, j = i / nin;
  const int k = (int)(i % nin), c = k / HW, pos = k % HW;
  Wc[j * nin + (long)pos * C + c] = W[i];
}

// Position of the k-th set bit (k counted from 0) of m, for k < popcount(m): a binary search
// over halves, quarters, ... of the word, by the popcount of each lower part (no branch).
__device__ __forceinline__ int kth_bit(unsigned m, int k) {
  int pos = 0;
#pragma unroll
  for (int w = 16; w >= 1; w >>= 1) {
    const unsigned low = m & ((1u << w) - 1u);
    const int c = __builtin_popcount(low);
    const bool up = k >= c;
    k = up ? k - c : k;
    pos += up ? w : 0;
    m = up ? m >> w : low;
  }
  return pos;
}

// Sum of v over the 8 rows of a position in k_fwd_conv12's layout: the lane's four rows are
// summed in place, then with the four rows of the lane 16 away (v_permlane16_swap exchanges rows
// 0 <-> 1 and 2 <-> 3 of 16 lanes; with the same value in both operands, the two results are
// the lane's own and its partner's value).
__device__ __forceinline__ float sum_rows8(const float4v& v) {
  const float own = (v[0] + v[1]) + (v[2] + v[3]);
  const auto sw = __builtin_amdgcn_permlane16_swap(__float_as_uint(own), __float_as_uint(own),
                                                   false, false);
  return __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
}

// The witness forward of a pass opened at a Linear layer T_3 over two convolutions
// T_1: Conv(3 -> C1, k4 s2 p1, 32x32 -> 16x16) and T_2: Conv(C1 -> C2, k4 s2 p1, 16x16 -> 8x8)
// (pass 3 of the Base and Wide nets), both layers in one kernel, with the adjoint sums of both
// layers fused.  One block (4 waves) takes one group of 8 rows q of the pass, which lie in one
// sub-domain (R is a multiple of 8).  It runs x* = x0 - eps sign(A_x) through T_1 (G_1, the
// adjoint terms of layer 1 against the recorded coefficients A~_1, then the row's relaxation
// line z_1), keeps z_1 in an LDS ring instead of writing it out, and runs z_1 through T_2 (G_2,
// the adjoint terms of layer 2 against A~_2 = +-W_3[j], the row's own coefficients).
// Both convolutions are gather-form implicit GEMMs on 16x16x4 MFMA with the activations as the
// A operand: M = the 8 rows at two output positions (m = 8 p + row), N = 16 output channels,
// one K step per (input channel, tap row) with the tap column as the lane group.  A lane then
// holds four rows (4 (g & 1) .. + 3, position g >> 1) of one output channel n: its adjoint
// terms are summed over the rows in place and once across lanes (sum_rows8), its z_1 values
// are one 16-byte LDS store, and its recorded coefficients one 16-byte read.
// Schedule over the output rows y2 of T_2: conv2 row y2 reads z_1 rows 2 y2 - 1 .. 2 y2 + 2
// (ring of 4 slots, row mod 4); then conv1 computes z_1 rows 2 y2 + 3 and 2 y2 + 4 into the two
// slots conv2 just finished with, from x* rows 4 y2 + 5 .. 4 y2 + 10 (ring of 6 slots, row
// mod 6).  While conv2 runs, the block fetches with coalesced 16-byte loads what conv1 will
// need -- the four new x* rows (signs and x0), and for its two rows the recorded coefficients
// A~_1 and the layer-1 relaxation -- and parks them in LDS.  The two tapes (the signs of A_x
// and A~_1, both written by k_convT_fc_bound) are blocked by groups of 8 rows,
// [q / 8][entry][q % 8], so the group's entries of a row are one contiguous run.  Rows outside
// a map are zero slots
// (the convolutions' zero padding).  Adjoint sums are written as k_fwd_conv writes them
// ([group][term][position][channel]); with 32 channels on T_2 the sums of both layers go only to
// the unstable neurons, by their rank in the sub-domain ([group][rank][term], k_grad_gather_c).  The LDS footprint lets two blocks share a CU, so one
// block's barriers overlap the other's work.  No load carries a per-lane condition (such a
// value makes the wave wait for it at once): out-of-map rows and rows past Q read clamped,
// in-bounds entries that are zeroed or meet a zero weight where they are used.
template <int C1, int C2>
__global__ void __launch_bounds__(256, 2)
    k_fwd_conv12(DLayer t1, DLayer t2, const int8_t* __restrict__ sgn, unsigned ldq, unsigned Q,
                 unsigned R, const float* __restrict__ w, const float* __restrict__ x0, float eps,
                 const float* __restrict__ tape1, const float* __restrict__ a_lo,
                 const float* __restrict__ a_up, const float* __restrict__ b_up,
                 unsigned pstride, const float* __restrict__ W3, unsigned nk, unsigned inter,
                 const unsigned* __restrict__ psel,
                 const int* __restrict__ kidx1, const int* __restrict__ kidx2,
                 const float* __restrict__ W2t,
                 float* __restrict__ part1,
                 float* __restrict__ part2,
                 unsigned char* __restrict__ gflag) {
  constexpr int C0 = 3, K = 4, S = 2, HX = 32, H1 = 16, H2 = 8;
  constexpr int N1 = C1 * H1 * H1, N2 = C2 * H2 * H2;
  constexpr int XW1 = (H1 - 1) * S + K;  // x* ring columns: x = -1 .. 32
  constexpr int XW2 = (H2 - 1) * S + K;  // z_1 ring columns: x1 = -1 .. 16
  // z_1 ring channel stride: 4 floats of padding put the 16-byte stores of the 16 channels of a
  // position on distinct banks
  constexpr int ZCS = XW2 * 8 + 4;
  constexpr int XROW = C0 * XW1 * 8, ZROW = C1 * ZCS;
  constexpr int NX = 6, NZ = 4;          // ring slots
  constexpr int NKS1 = C0 * K, NKS2 = C1 * K;
  constexpr int NMT2 = C2 / 16;          // channel tiles of T_2
  static_assert(C1 == 8 || C1 == 16, "T_1 output channels");
  static_assert(C2 == 16 || C2 == 32, "T_2 output channels");
  // With 32 channels, conv2 runs only where its adjoint terms are used: at the layer-2 neurons
  // that are unstable in the block's sub-domain.  The 8 positions of a row are paired, the one
  // with the most unstable channels with the one with the fewest and so on (so that a pair
  // rarely has more than 16), and wave w takes pair w; the channels unstable at either position
  // of its pair are packed into tiles of 16 (one tile for up to 16 such channels, two above),
  // and lane n of a tile computes the n-th of them.  W3 is then the channel-last copy of W_3
  // (k_fc_chlast), whose entries of one position are contiguous.
  constexpr bool GATHER = C2 == 32;
  // conv1 epilogue operands of the two rows of an iteration: relaxation [row][a_lo, a_up, b_up]
  // [x1][channel] and coefficients [row][x1][channel][q]
  // (GATHER: a fourth, the neuron's rank among the sub-domain's unstable layer-1 neurons, or -1,
  // staged as 16 bits in ep_k, so that two blocks still share a CU)
  constexpr int NPR = GATHER ? 4 : 3;
  constexpr int EPP = 2 * 3 * H1 * C1, EPT = 2 * H1 * C1 * 8;
  __shared__ __attribute__((aligned(16))) float xr[NX * XROW];
  __shared__ __attribute__((aligned(16))) float zr[NZ * ZROW];
  __shared__ float ep_p[EPP];
  __shared__ short ep_k[GATHER ? 2 * H1 * C1 : 1];
  __shared__ __attribute__((aligned(16))) float ep_t[EPT];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 15, g = lane >> 4;
  const int qr = n & 7, pp = n >> 3;  // A operand: this lane's row and position of a pair
  const int qb = 4 * (g & 1), pd = g >> 1;  // D: this lane's first row and position
  const unsigned grp = xcd_range(blockIdx.x);
  const unsigned q0 = grp * 8u;
  if (q0 >= Q) return;  // grid padding, uniform per block
  // the lane's four D rows: weight, sign and row of W_3 of each (rows past Q: weight 0)
  float wq[4], tsg[4];
  const float* w3r[4];
  bool any = false;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const unsigned q = q0 + qb + r;
    const bool ok = q < Q;
    wq[r] = ok ? w[min(q, Q - 1)] : 0.f;
    // row ra of the sub-domain: +-e_j, the signs in two halves or interleaved (inter)
    const unsigned ra = q % R;
    const bool neg = inter ? (ra & 1u) != 0 : ra >= nk;
    tsg[r] = !ok ? 0.f : (neg ? -1.f : 1.f);
    w3r[r] = W3 + (size_t)(inter ? ra >> 1 : ra % nk) * N2;
    any |= wq[r] != 0.f;
  }
  {
    const bool live = __syncthreads_or(any) != 0;
    if (tid == 0) gflag[grp] = live ? 1 : 0;
    if (!live) return;  // uniform: the whole block is idle
  }
  const unsigned b = q0 / R;  // the group's sub-domain
  const int mt2 = wave % NMT2;

  // B operands: lane (n, g) holds W[co = n][ci][ky][kx = g] per K step (ci, ky); the bias of
  // this lane's output channel.  (GATHER: the conv2 operands of the wave's next tile, loaded
  // per tile.)
  float w1r[NKS1], w2r[NKS2];
#pragma unroll
  for (int ks = 0; ks < NKS1; ++ks)
    w1r[ks] = n < C1 ? t1.W[((n * C0 + ks / K) * K + ks % K) * K + g] : 0.f;
  if constexpr (!GATHER) {
#pragma unroll
    for (int ks = 0; ks < NKS2; ++ks)
      w2r[ks] = t2.W[(((mt2 * 16 + n) * C1 + ks / K) * K + ks % K) * K + g];
  }
  const float b1 = n < C1 ? t1.b[n] : 0.f;
  int co2 = mt2 * 16 + n;
  float b2 = GATHER ? 0.f : t2.b[co2];
  // (GATHER: a lane past the tile's last channel repeats that channel, computes the same
  // values and stores them to the same place)
  // tile t of mask m (row y2): this lane's channel and bias, its conv2 operands and its
  // coefficients over g^(2).  Lane group g = kx loads the four taps ky = 0..3 of tap column g of
  // each input channel as one 16-byte quad of the tap-swapped weights, which are the operands
  // of K steps (ci, ky) in registers 4 ci + ky.
  float4v tw;
  // (k2: the rank of the lane's layer-2 neuron among the sub-domain's unstable ones, or -1)
  int k2 = -1, k2n = -1;
  auto tile_load = [&](unsigned m, int t, int y2, int xa, int xb) {
    const int cnt = __builtin_popcount(m);
    const int k = n + 16 * t;
    co2 = kth_bit(m, min(k, cnt - 1));
    b2 = t2.b[co2];
    const float4v* wp = reinterpret_cast<const float4v*>(W2t + (size_t)co2 * (C1 * K * K)) + g;
#pragma unroll
    for (int ci = 0; ci < C1; ++ci) {
      const float4v v = wp[ci * K];
#pragma unroll
      for (int j = 0; j < 4; ++j) w2r[ci * K + j] = v[j];
    }
    const int o = (y2 * H2 + (pd ? xb : xa)) * C2 + co2;
#pragma unroll
    for (int r = 0; r < 4; ++r) tw[r] = w3r[r][o];  // (times the row's sign where used)
    k2 = kidx2[(size_t)b * N2 + (co2 * H2 + y2) * H2 + (pd ? xb : xa)];
  };
  // the tile after the current one: its channel, bias and coefficients now, its conv2 operands
  // (from the returned quads) one input channel at a time during the current tile's MFMAs, into
  // the registers those MFMAs have just read, so that the loads overlap the MFMA chain
  int co2n = 0;
  float b2n = 0.f;
  float4v twn;
  auto next_setup = [&](unsigned m, int t, int y2, int xa, int xb) {
    const int cnt = __builtin_popcount(m);
    const int k = n + 16 * t;
    co2n = kth_bit(m, min(k, cnt - 1));
    b2n = t2.b[co2n];
    const int o = (y2 * H2 + (pd ? xb : xa)) * C2 + co2n;
#pragma unroll
    for (int r = 0; r < 4; ++r) twn[r] = w3r[r][o];
    k2n = kidx2[(size_t)b * N2 + (co2n * H2 + y2) * H2 + (pd ? xb : xa)];
    return reinterpret_cast<const float4v*>(W2t + (size_t)co2n * (C1 * K * K)) + g;
  };
  // each row's pair of positions (xa | xb << 3) for this wave and the channels unstable at
  // either of them (wave-uniform, k_pair_select), kept in LDS
  __shared__ unsigned gsel[GATHER ? 4 : 1][H2][2];
  if constexpr (GATHER) {
    if (lane < 2 * H2) (&gsel[wave][0][0])[lane] = psel[((size_t)b * 4 + wave) * (2 * H2) + lane];
  }

  auto xslot = [](int yi) { return (yi + 6 * NX) % NX; };
  auto zslot = [](int y1) { return (y1 + 4 * NZ) % NZ; };

  // pad columns of every slot, and the z_1 row -1 (slot 3), are zero for good
  for (int e = tid; e < NX * C0 * 2 * 8; e += 256) {
    const int qq = e & 7, side = (e >> 3) & 1, sc = e >> 4;
    xr[(sc * XW1 + (side ? XW1 - 1 : 0)) * 8 + qq] = 0.f;
  }
  for (int e = tid; e < NZ * C1 * 2 * 8; e += 256) {
    const int qq = e & 7, side = (e >> 3) & 1, sc = e >> 4;
    zr[sc * ZCS + (side ? XW2 - 1 : 0) * 8 + qq] = 0.f;
  }
  for (int e = tid; e < ZROW; e += 256) zr[zslot(-1) * ZROW + e] = 0.f;

  // x* rows, 4 at a time: element e = (row j, channel ci, column x, half h of the 8 rows); the
  // signs of 4 rows are one 32-bit word of the byte tape
  constexpr int NXE = 4 * C0 * HX * 2;
  constexpr int XPT = NXE / 256;
  static_assert(NXE % 256 == 0, "whole x* elements per thread");
  int sw[XPT];
  float sx[XPT];
  auto fetch_x = [&](int yfirst) {
#pragma unroll
    for (int k = 0; k < XPT; ++k) {
      const int e = tid + k * 256;
      const int h = e & 1, x = (e >> 1) % HX, ci = (e >> 1) / HX % C0;
      const int yc = min(max(yfirst + e / (2 * C0 * HX), 0), HX - 1);
      sw[k] = *reinterpret_cast<const int*>(
          sgn + (size_t)(q0 / 8) * (C0 * HX * HX * 8) + (size_t)((ci * HX + yc) * HX + x) * 8 +
          4 * h);
      sx[k] = x0[(ci * HX + yc) * HX + x];
    }
  };
  auto park_x = [&](int yfirst) {
#pragma unroll
    for (int k = 0; k < XPT; ++k) {
      const int e = tid + k * 256;
      const int h = e & 1, x = (e >> 1) % HX, ci = (e >> 1) / HX % C0;
      const int yi = yfirst + e / (2 * C0 * HX);
      const bool in = yi >= 0 && yi < HX;
      float4v v;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        v[jj] = in ? sx[k] - eps * (float)(int8_t)(sw[k] >> (8 * jj)) : 0.f;
      *reinterpret_cast<float4v*>(xr + ((xslot(yi) * C0 + ci) * XW1 + x + 1) * 8 + 4 * h) = v;
    }
  };
  // conv1 epilogue operands of rows ya, ya + 1 (a row past the map reads row H1 - 1: unused):
  // relaxation element e = (row, param, quad of x1, channel), coefficient element
  // e = (row, x1, channel, half of the 8 rows q), each one 16-byte load; consecutive threads
  // take consecutive channels, so that their LDS stores fall on distinct banks
  constexpr int NPE = 2 * NPR * 4 * C1, NTE = 2 * H1 * C1 * 2;
  constexpr int PPT = (NPE + 255) / 256, TPT = NTE / 256;
  static_assert(NTE % 256 == 0, "whole coefficient elements per thread");
  float4v pv[PPT], tv[TPT];
  // this thread's relaxation array per element (a_lo, a_up or b_up), chosen once: a per-lane
  // pointer select in the loop compiles to branches
  const float* psrc[PPT];
#pragma unroll
  for (int k = 0; k < PPT; ++k) {
    const int e = min(tid + k * 256, NPE - 1);
    const int pr = e / (4 * C1) % NPR;
    psrc[k] = pr == 3 ? reinterpret_cast<const float*>(kidx1) + (size_t)b * N1
                      : (pr == 0 ? a_lo : (pr == 1 ? a_up : b_up)) + (size_t)b * pstride;
  }
  auto fetch_ep = [&](int ya) {
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
      const int e = min(tid + k * 256, NPE - 1);
      const int c = e % C1, x4 = (e / C1) & 3, r2 = e / (4 * C1 * NPR);
      const int y1 = min(ya + r2, H1 - 1);
      pv[k] = *reinterpret_cast<const float4v*>(psrc[k] + (c * H1 + y1) * H1 + 4 * x4);
    }
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
      const int e = tid + k * 256;
      const int h = e & 1, c = (e >> 1) % C1, x1 = (e >> 1) / C1 % H1, r2 = e / (2 * H1 * C1);
      const int y1 = min(ya + r2, H1 - 1);
      tv[k] = *reinterpret_cast<const float4v*>(
          tape1 + (size_t)(q0 / 8) * (N1 * 8) + (size_t)((c * H1 + y1) * H1 + x1) * 8 + 4 * h);
    }
  };
  auto park_ep = [&]() {
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
      const int e = tid + k * 256;
      if (NPE % 256 == 0 || e < NPE) {
        const int c = e % C1, x4 = (e / C1) & 3, pr = e / (4 * C1) % NPR,
                  r2 = e / (4 * C1 * NPR);
        if (GATHER && pr == 3) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            ep_k[(r2 * H1 + 4 * x4 + i) * C1 + c] = (short)__float_as_int(pv[k][i]);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) ep_p[((r2 * 3 + pr) * H1 + 4 * x4 + i) * C1 + c] = pv[k][i];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
      const int e = tid + k * 256;
      const int h = e & 1, c = (e >> 1) % C1, x1 = (e >> 1) / C1 % H1, r2 = e / (2 * H1 * C1);
      *reinterpret_cast<float4v*>(ep_t + ((r2 * H1 + x1) * C1 + c) * 8 + 4 * h) = tv[k];
    }
  };

  // one T_1 position pair (row y1 = ya + r2, columns 2 xp, 2 xp + 1)
  auto conv1_pos = [&](int y1, int r2, int xp) {
    const float* xb[K];
#pragma unroll
    for (int ky = 0; ky < K; ++ky)
      xb[ky] = xr + xslot(2 * y1 - 1 + ky) * XROW + (2 * (2 * xp + pp) + g) * 8 + qr;
    float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < NKS1; ++ks)
      d = __builtin_amdgcn_mfma_f32_16x16x4f32(xb[ks % K][(ks / K) * XW1 * 8], w1r[ks], d, 0, 0,
                                               0);
    const int x1 = 2 * xp + pd;
    const int c = min(n, C1 - 1);  // (lanes of channels past C1 read a valid entry, unused)
    const float4v tt = *reinterpret_cast<const float4v*>(ep_t + ((r2 * H1 + x1) * C1 + c) * 8 + qb);
    const float lo = ep_p[((r2 * 3 + 0) * H1 + x1) * C1 + c];
    const float up = ep_p[((r2 * 3 + 1) * H1 + x1) * C1 + c];
    const float bu = ep_p[((r2 * 3 + 2) * H1 + x1) * C1 + c];
    float4v ta, tb, tc, z;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float gv = d[r] + b1;
      // a row without weight (rows past Q included) gets zero terms and z_1 = 0
      const float t = wq[r] != 0.f ? tt[r] : 0.f;
      const float tp = fmaxf(t, 0.f), tn = fminf(t, 0.f);
      ta[r] = (wq[r] * tp) * gv;
      tb[r] = (wq[r] * tn) * gv;
      tc[r] = wq[r] * tn;
      // both lines computed and selected (no branch): the z_1 of a row without weight is 0
      const float zl = lo * gv, zu = fmaf(up, gv, bu);
      const float zs = t >= 0.f ? zl : zu;
      z[r] = wq[r] != 0.f ? zs : 0.f;
    }
    if (n < C1)
      *reinterpret_cast<float4v*>(zr + zslot(y1) * ZROW + n * ZCS + (x1 + 1) * 8 + qb) = z;
    const float sa = sum_rows8(ta), da = sum_rows8(tb), db = sum_rows8(tc);
    if constexpr (GATHER) {
      // only the unstable neurons' sums are used: at the neuron's rank in the sub-domain,
      // [group][rank][3] (k_grad_gather_c)
      const int kr = ep_k[(r2 * H1 + x1) * C1 + c];
      if ((g & 1) == 0 && kr >= 0) {
        float* dst = part1 + ((size_t)grp * N1 + kr) * 3;
        dst[0] = sa;
        dst[1] = da;
        dst[2] = db;
      }
    } else if ((g & 1) == 0 && n < C1) {
      float* dst = part1 + (size_t)grp * 3 * N1 + (size_t)(y1 * H1 + x1) * C1 + n;
      dst[0] = sa;
      dst[N1] = da;
      dst[2 * N1] = db;
    }
  };
  // a T_1 row: 8 position pairs, pairs wave and wave + 4
  auto conv1_row = [&](int y1, int r2) {
    if (y1 >= H1) {
      // the z_1 row below the map: zeros
      for (int e2 = tid; e2 < ZROW; e2 += 256) zr[zslot(y1) * ZROW + e2] = 0.f;
      return;
    }
    conv1_pos(y1, r2, wave);
    conv1_pos(y1, r2, wave + 4);
  };
  // a T_2 row: 4 position pairs times NMT2 channel tiles, NMT2 per wave
  constexpr int P2W = NMT2;
  auto xp2 = [&](int k) { return wave / NMT2 + k * (4 / NMT2); };
  // this lane's entries of the rows' coefficients over g^(2), +-W_3[j] at (co2, y2, x2)
  auto load_tw = [&](int y2, float4v* tw) {
#pragma unroll
    for (int k = 0; k < P2W; ++k) {
      const int o = (co2 * H2 + y2) * H2 + 2 * xp2(k) + pd;
#pragma unroll
      for (int r = 0; r < 4; ++r) tw[k][r] = tsg[r] * w3r[r][o];
    }
  };
  // a T_2 position pair (xa, xb) of row y2 (A operand rows 0..7 at xa, 8..15 at xb)
  // (GATHER: wpn, the next tile's operand quads, loaded into w2r as its entries are used)
  auto conv2_pos = [&](int y2, int xa, int xb, const float4v& tw, const float4v* wpn) {
    const float* zb[K];
#pragma unroll
    for (int ky = 0; ky < K; ++ky)
      zb[ky] = zr + zslot(2 * y2 - 1 + ky) * ZROW + (2 * (pp ? xb : xa) + g) * 8 + qr;
    float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ci = 0; ci < C1; ++ci) {
#pragma unroll
      for (int ky = 0; ky < K; ++ky)
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(zb[ky][ci * ZCS], w2r[ci * K + ky], d, 0, 0, 0);
      if constexpr (GATHER) {
        const float4v v = wpn[ci * K];
#pragma unroll
        for (int j = 0; j < 4; ++j) w2r[ci * K + j] = v[j];
        // (keep each load behind the four MFMAs that free its registers, not bunched at the end)
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
    }
    float4v ta, tb, tc;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float gv = d[r] + b2;
      const float tp = fmaxf(tw[r], 0.f), tn = fminf(tw[r], 0.f);
      ta[r] = (wq[r] * tp) * gv;
      tb[r] = (wq[r] * tn) * gv;
      tc[r] = wq[r] * tn;
    }
    const float sa = sum_rows8(ta), da = sum_rows8(tb), db = sum_rows8(tc);
    if constexpr (GATHER) {
      // the unstable neurons' sums at their ranks, [group][rank][3], as the layer-1 sums
      if ((g & 1) == 0 && k2 >= 0) {
        float* dst = part2 + ((size_t)grp * N2 + k2) * 3;
        dst[0] = sa;
        dst[1] = da;
        dst[2] = db;
      }
    } else if ((g & 1) == 0) {
      const int x2 = pd ? xb : xa;
      float* dst = part2 + (size_t)grp * 3 * N2 + (size_t)(y2 * H2 + x2) * C2 + co2;
      dst[0] = sa;
      dst[N2] = da;
      dst[2 * N2] = db;
    }
  };

  // prologue: z_1 row 0 (epilogue operands of rows 0, 1), then rows 1, 2
  if constexpr (GATHER) {
    const unsigned m0 = __builtin_amdgcn_readfirstlane(gsel[wave][0][0]);
    const unsigned s0 = __builtin_amdgcn_readfirstlane(gsel[wave][0][1]);
    tile_load(m0, 0, 0, s0 & 7, s0 >> 3);
  }
  fetch_x(-1);
  fetch_ep(0);
  park_x(-1);
  park_ep();
  __syncthreads();
  conv1_row(0, 0);
  fetch_x(3);
  __syncthreads();  // x* row 0's slot is free
  park_x(3);
  __syncthreads();
  conv1_row(1, 1);
  fetch_ep(2);
  __syncthreads();  // the staged operands of rows 0, 1 are consumed
  park_ep();
  // the operands of the first iteration's conv1 rows: in flight during row 2 and conv2 row 0
  fetch_x(7);
  fetch_ep(3);
  __syncthreads();
  conv1_row(2, 0);
  __syncthreads();

  for (int y2 = 0; y2 < H2; ++y2) {
    const int ya = 2 * y2 + 3, yb = 2 * y2 + 4;  // z_1 rows this iteration adds
    const bool more = ya < H1 + 1;               // (row 16 is the zero row)
    if constexpr (GATHER) {
      const unsigned umask = __builtin_amdgcn_readfirstlane(gsel[wave][y2][0]);
      const unsigned sel = __builtin_amdgcn_readfirstlane(gsel[wave][y2][1]);
      const int xa = sel & 7, xb = sel >> 3;
      // tile 0 always runs (with no unstable channel it computes channel 0, which no one
      // reads), so that the code from here to the barrier has no branch around a memory
      // operation and its memory waits count exactly the operations before them
      const bool two = __builtin_popcount(umask) > 16;
      const int yn = min(y2 + 1, H2 - 1);  // (the last row fetches its own first tile again)
      const unsigned un = __builtin_amdgcn_readfirstlane(gsel[wave][yn][0]);
      const unsigned sn = __builtin_amdgcn_readfirstlane(gsel[wave][yn][1]);
      auto tile = [&](const float4v* wpn) {
        float4v tws;
#pragma unroll
        for (int r = 0; r < 4; ++r) tws[r] = tsg[r] * tw[r];
        conv2_pos(y2, xa, xb, tws, wpn);
        co2 = co2n;
        b2 = b2n;
        tw = twn;
        k2 = k2n;
      };
      {
        // the tile after this one: the row's second, else the next row's first
        const unsigned mn = two ? umask : un, snx = two ? sel : sn;
        tile(next_setup(mn, two ? 1 : 0, two ? y2 : yn, snx & 7, snx >> 3));
      }
      if (two) {
        // (the tiles of a pair share their A operands: a compiler barrier keeps them read per
        // tile rather than held in registers across the tiles)
        asm volatile("" ::: "memory");
        tile(next_setup(un, 0, yn, sn & 7, sn >> 3));
      }
    } else {
      float4v tw[P2W];
      load_tw(y2, tw);
#pragma unroll
      for (int k = 0; k < P2W; ++k) conv2_pos(y2, 2 * xp2(k), 2 * xp2(k) + 1, tw[k], nullptr);
    }
    if (!more) break;
    park_x(4 * y2 + 7);
    park_ep();
    // the next iteration's operands: in flight during this iteration's conv1 and the next conv2
    if (ya + 2 < H1 + 1) {
      fetch_x(4 * y2 + 11);
      fetch_ep(ya + 2);
    }
    __syncthreads();  // staged rows visible; every wave is done with the z_1 slots it overwrites
    conv1_row(ya, 0);
    conv1_row(yb, 1);
    __syncthreads();  // z_1 rows visible to the next conv2 row; staged operands consumed
  }
}

// The unstable neurons of a layer, numbered per sub-domain in neuron order: kidx[b][j] = the
// rank of neuron j among the sub-domain's unstable neurons (-1 if it is not unstable),
// list[b][k] = the neuron of rank k, cnt[b] = their number.  One block per sub-domain.
__global__ void __launch_bounds__(256)
    k_unstable_index(int n, const int8_t* __restrict__ code, long n_relu, int* __restrict__ kidx,
                     int* __restrict__ list, int* __restrict__ cnt) {
  __shared__ int wsum[4];
  const long b = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int base = 0;
  for (int j0 = 0; j0 < n; j0 += 256) {
    const int j = j0 + threadIdx.x;
    const bool un = j < n && code[b * n_relu + j] == 5;
    const unsigned long long m = __ballot(un);
    const int below = (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
    if (lane == 0) wsum[wave] = __popcll(m);
    __syncthreads();
    int off = base;
    for (int w = 0; w < wave; ++w) off += wsum[w];
    const int k = off + below;
    if (j < n) kidx[b * n + j] = un ? k : -1;
    if (un) list[b * n + k] = j;
    base += wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();  // wsum is rewritten by the next chunk
  }
  if (threadIdx.x == 0) cnt[b] = base;
}

// The position pairs of k_fwd_conv12's layer-2 tiles (T_2 with 32 channels on an 8 x 8 map), the
// same for every group of rows of a sub-domain, so found once per sub-domain: for wave w of that
// kernel and map row y, sel[b][w][y] = (the channels unstable at either position of the wave's
// pair, xa | xb << 3).  The 8 positions of a row are ranked by (number of unstable channels,
// position) and wave w takes ranks w and 7 - w.  One block of 4 waves per sub-domain, wave w
// for pairs w; the stability codes are read once (lane c and c + 32 read channel c of two rows,
// one byte per position) and counted by ballot.
__global__ void __launch_bounds__(256)
    k_pair_select(const int8_t* __restrict__ code2, unsigned n_relu, unsigned* __restrict__ sel) {
  constexpr int H2 = 8;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned b = blockIdx.x;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int8_t* cc = code2 + (size_t)b * n_relu + (lane & 31) * (H2 * H2) + (lane >> 5) * H2;
  int8_t cd[H2 / 2][H2];
#pragma unroll
  for (int yy = 0; yy < H2 / 2; ++yy)
#pragma unroll
    for (int x = 0; x < H2; ++x) cd[yy][x] = cc[2 * yy * H2 + x];
  unsigned* out = sel + ((size_t)b * 4 + wv) * (2 * H2);
#pragma unroll
  for (int yy = 0; yy < H2 / 2; ++yy) {
    unsigned m[2][H2];
#pragma unroll
    for (int x = 0; x < H2; ++x) {
      const unsigned long long bm = __ballot(cd[yy][x] == 5);
      m[0][x] = (unsigned)bm;
      m[1][x] = (unsigned)(bm >> 32);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // rank of each position by (count, position); this wave's pair: ranks wv and 7 - wv
      int key[H2];
#pragma unroll
      for (int x = 0; x < H2; ++x) key[x] = __builtin_popcount(m[h][x]) * H2 + x;
      int xa = 0, xb = 0;
      unsigned ma = 0u, mb = 0u;
#pragma unroll
      for (int x = 0; x < H2; ++x) {
        int rk = 0;
#pragma unroll
        for (int x2 = 0; x2 < H2; ++x2) rk += key[x2] < key[x] ? 1 : 0;
        xa = rk == wv ? x : xa;
        ma = rk == wv ? m[h][x] : ma;
        xb = rk == H2 - 1 - wv ? x : xb;
        mb = rk == H2 - 1 - wv ? m[h][x] : mb;
      }
      if (lane == 0) {
        out[(2 * yy + h) * 2] = ma | mb;
        out[(2 * yy + h) * 2 + 1] = (unsigned)xa | ((unsigned)xb << 3);
      }
    }
  }
}

// k_grad_gather over compacted partial sums: part[(b (R / 8) + k8) n_m + k][3] holds the sums of
// the unstable neuron of rank k (k_unstable_index) for group k8 of sub-domain b.  A block per
// sub-domain, a thread per rank: the same sums in the same group order as k_grad_gather, from
// contiguous memory.
__global__ void __launch_bounds__(kBlock)
    k_grad_gather_c(long nm, long R, const float* __restrict__ part,
                    const unsigned char* __restrict__ gflag, const int* __restrict__ list,
                    const int* __restrict__ cnt, const float* __restrict__ l,
                    const float* __restrict__ u, long n_relu, float* __restrict__ ga,
                    float* __restrict__ gl, float* __restrict__ gu) {
  const long b = blockIdx.x;
  const int nk = cnt[b];
  const long ng = R / 8, g0 = b * ng;
  for (int k = threadIdx.x; k < nk; k += blockDim.x) {
    const long p = b * n_relu + list[b * nm + k];
    // (flags as in k_grad_gather)
    float sa = 0.f, da = 0.f, db = 0.f;
    const float* src = part + (g0 * nm + k) * 3;
#pragma unroll 5
    for (long k8 = 0; k8 < ng; ++k8) {
      const bool on = gflag[g0 + k8] != 0;
      const float* e = src + k8 * nm * 3;
      const float a0 = e[0], a1 = e[1], a2 = e[2];
      sa += on ? a0 : 0.f;
      da += on ? a1 : 0.f;
      db += on ? a2 : 0.f;
    }
    const float lj = l[p], uj = u[p], dd = uj - lj, d2 = dd * dd;
    ga[p] += sa;
    gl[p] += (da * uj - db * uj * uj) / d2;
    gu[p] += (-da * lj + db * lj * lj) / d2;
  }
}

// Adjoint accumulation for ReLU layer m from the partial sums of the fused witness forward: for
// each (sub-domain, neuron), the R/8 groups of 8 rows of the sub-domain in increasing order (an
// order fixed by the rows alone, so the result does not depend on where the sub-domain sits in
// the chunk), skipping groups without weight; then, for unstable neurons, as k_grad_reduce.
// Threads run over (sub-domain, position, channel) with the channel fastest, the order of the
// partial sums.
__global__ void __launch_bounds__(kBlock)
    k_grad_gather(long nb, int CO, int NPOS, long R, const float* __restrict__ part,
                  const unsigned char* __restrict__ gflag, const int8_t* __restrict__ code,
                  const float* __restrict__ l, const float* __restrict__ u, long n_relu,
                  float* __restrict__ ga, float* __restrict__ gl, float* __restrict__ gu) {
  const long nm = (long)CO * NPOS;
  const long idx = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (idx >= nb * nm) return;
  const long b = idx / nm, oc = idx % nm;
  const int pos = (int)(oc / CO), co = (int)(oc % CO);
  const long j = (long)co * NPOS + pos;
  const long p = b * n_relu + j;
  if (code[p] != 5) return;
  const long g0 = b * (R / 8), ng = R / 8;
  // every group's entries are loaded (in bounds, possibly stale where the group had no weight)
  // and a group without weight adds nothing: no load waits for a flag, so the loads of several
  // groups are in flight together
  float sa = 0.f, da = 0.f, db = 0.f;
#pragma unroll 5
  for (long k = 0; k < ng; ++k) {
    const bool on = gflag[g0 + k] != 0;
    const float* src = part + (g0 + k) * 3 * nm + oc;
    const float a0 = src[0], a1 = src[nm], a2 = src[2 * nm];
    sa += on ? a0 : 0.f;
    da += on ? a1 : 0.f;
    db += on ? a2 : 0.f;
  }
  const float lj = l[p], uj = u[p], dd = uj - lj, d2 = dd * dd;
  ga[p] += sa;
  gl[p] += (da * uj - db * uj * uj) / d2;
  gu[p] += (-da * lj + db * lj * lj) / d2;
}

// The witness forward step through a convolution of a covered shape (k <= 4), as a gather-form
// implicit GEMM on 16x16x4 MFMA: M = 16 output channels, N = 16 rows q, and one K step per
// (input channel ci, tap row ky) whose four K entries are the tap columns kx = lane group (a
// column kx >= k carries a zero weight), so the input row and channel of a K step are uniform
// over the wave.  Output rows are visited in order; the input rows they need sit in an LDS ring
// ([slot][ci][x][16 rows q], slot = input row mod NSLOT, zero rows for the padding), and the S
// input rows the next output row adds are loaded into registers at the start of a row and parked
// in the ring after its MFMAs (with WITNESS, turned into x0 - eps sign(A_x) on the way).  Each
// wave owns one M tile (16 output channels) and holds all its A operands (weights) in registers;
// the output positions of a row are dealt to the waves of an M tile.  Epilogue: G =
// pre-activation, zout = the row's relaxation line applied, or the fused adjoint sums.
template <int K, int S, int P, int CI, int CO, int HI, int WI, int HO, int WO, bool WITNESS,
          bool ZOUT>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(
    ZOUT ? (CI * K >= 64 ? 2 : (CI * K >= 24 ? 3 : 4)) : (CI * K >= 64 ? 3 : 4), 8)))
    k_fwd_conv(DLayer t, const float* __restrict__ zin, unsigned ldq, unsigned Q, long R,
               const float* __restrict__ w, const float* __restrict__ x0, float eps,
               const float* __restrict__ tape, const float* __restrict__ a_lo,
               const float* __restrict__ a_up, const float* __restrict__ b_up, long pstride,
               float* __restrict__ G, float* __restrict__ zout, float* __restrict__ part,
               unsigned char* __restrict__ gflag, const float* __restrict__ tapeW, int tnk,
               int ns) {
  static_assert(K <= 4, "tap columns are the four lane groups");
  constexpr int NKS = CI * K;                // K steps
  constexpr int NMT = (CO + 15) / 16;        // M tiles
  static_assert(NMT == 1 || NMT == 2 || NMT == 4, "M tiles are dealt to the 4 waves");
  constexpr int NPOS = HO * WO;
  constexpr int PSTEP = 4 / NMT;             // waves per M tile
  static_assert(WO % PSTEP == 0, "the positions of a row are dealt evenly");
  constexpr int IPW = WO / PSTEP;            // positions per wave and output row
  // a ring row holds the input columns -P .. (WO-1)*S - P + 3 (zero outside the map), so every
  // lane's column of every K step is in range and needs no test
  constexpr int XW = (WO - 1) * S + 4;
  static_assert(P >= 0 && P + WI <= XW, "ring row covers the map");
  constexpr int ROWF = CI * XW * 16;         // floats of one input row in the ring
  // K + S slots (one barrier per output row) where they fit in 48 KB, else K (two barriers)
  constexpr int NSLOT = (K + S) * ROWF * 4 <= 48 * 1024 ? K + S : K;
  constexpr bool TWO_BAR = NSLOT == K;
  constexpr int NF4 = S * CI * WI * 4;       // float4 of the S input rows an output row adds
  constexpr int PFT = (NF4 + 255) / 256;
  static_assert(K % S == 0 || !TWO_BAR, "prologue chunks fit the ring");
  __shared__ float xs[WITNESS ? CI * HI * WI : 1];
  __shared__ float ring[NSLOT * ROWF];
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int n = lane & 15, g = lane >> 4;
  // ns = 2: two blocks per 16-row tile, each over half of the output rows (more blocks for a
  // small batch of rows)
  const unsigned q0 = xcd_tile(ns == 2 ? blockIdx.x >> 1 : blockIdx.x) * 16u;
  const int y_lo = ns == 2 ? (int)(blockIdx.x & 1u) * (HO / 2) : 0;
  const int y_hi = ns == 2 ? y_lo + HO / 2 : HO;
  if (q0 >= Q) return;  // grid padding, uniform per block
  const unsigned q = q0 + n;
  const bool qok = q < Q;
  const float wq = qok ? w[q] : 0.f;
  if (part) {
    // the two groups of 8 rows of this tile: does any row carry weight
    const bool live = __syncthreads_or(wq != 0.f && n < 8) != 0;
    const bool live2 = __syncthreads_or(wq != 0.f && n >= 8) != 0;
    if (threadIdx.x == 0) {
      gflag[q0 / 8] = live ? 1 : 0;
      gflag[q0 / 8 + 1] = live2 ? 1 : 0;
    }
  }
  if (__syncthreads_or(wq != 0.f) == 0) return;  // uniform: the whole block is idle
  const unsigned b = qok ? q / (unsigned)R : 0u;
  const int mt = wave % NMT;
  float wreg[NKS];
  {
    const int co = mt * 16 + n;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int ci = ks / K, ky = ks % K;
      wreg[ks] = (co < CO && g < K) ? t.W[((co * CI + ci) * K + ky) * K + g] : 0.f;
    }
  }
  if constexpr (WITNESS) {
    for (int e = threadIdx.x; e < CI * HI * WI; e += 256) xs[e] = x0[e];
    __syncthreads();
  }

  // input rows ybase .. ybase+S-1 into registers (float4 e = (row j, ci, x, quarter of q))
  auto slot_of = [](int yi) { return (yi + 8 * NSLOT) % NSLOT; };
  // (WITNESS: the four rows' signs of the sign tape, one 32-bit word, in pf[k][0])
  float4v pf[PFT];
  auto fetch_rows = [&](int ybase) {
#pragma unroll
    for (int k = 0; k < PFT; ++k) {
      const int e = threadIdx.x + k * 256;
      pf[k] = float4v{0.f, 0.f, 0.f, 0.f};
      if (e < NF4) {
        const int j4 = e & 3, fr = e >> 2;
        const int xi = fr % WI, ci = (fr / WI) % CI, yi = ybase + fr / (WI * CI);
        if (yi >= 0 && yi < HI) {
          const size_t at = (size_t)(((unsigned)ci * HI + yi) * WI + xi) * ldq + q0 + 4 * j4;
          if constexpr (WITNESS)
            pf[k][0] = __builtin_bit_cast(
                float, *reinterpret_cast<const int*>(reinterpret_cast<const int8_t*>(zin) + at));
          else
            pf[k] = *reinterpret_cast<const float4v*>(zin + at);
        }
      }
    }
  };
  // ... and into their ring slots (rows outside the map stay zero)
  auto park_rows = [&](int ybase) {
#pragma unroll
    for (int k = 0; k < PFT; ++k) {
      const int e = threadIdx.x + k * 256;
      if (e < NF4) {
        const int j4 = e & 3, fr = e >> 2;
        const int xi = fr % WI, ci = (fr / WI) % CI, yi = ybase + fr / (WI * CI);
        float4v v = pf[k];
        if constexpr (WITNESS) {
          if (yi >= 0 && yi < HI) {
            const float xv = xs[((unsigned)ci * HI + yi) * WI + xi];
            const int sw = __builtin_bit_cast(int, pf[k][0]);
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
              v[jj] = xv - eps * (float)(int8_t)(sw >> (8 * jj));
          }
        }
        *reinterpret_cast<float4v*>(ring + ((slot_of(yi) * CI + ci) * XW + xi + P) * 16 + 4 * j4) =
            v;
      }
    }
  };
  // epilogue operands of an output position (tape and relaxation line of the 4 outputs of this
  // lane), fetched one position ahead when there is a next layer to feed
  // (ZOUT: the output feeds a next layer; part: the adjoint sums are fused)
  const bool fz = (ZOUT || part != nullptr) && qok && wq != 0.f;
  constexpr int NE = ZOUT ? 4 : 1;
  float et[4], el[NE], eu[NE], eb[NE];
  auto load_ep = [&](int p_, float* t_, float* l_, float* u_, float* b_) {
    const int y = p_ / WO, x = p_ - y * WO;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int co = mt * 16 + 4 * g + r;
      t_[r] = 0.f;
      if constexpr (ZOUT) l_[r] = u_[r] = b_[r] = 0.f;
      if (fz && co < CO) {
        const unsigned o = ((unsigned)co * HO + y) * WO + x;
        if (tapeW) {
          // the pass's rows over this layer's output are +-W_k[j] (j = r mod nk, sign + for
          // r < nk): no recorded tape
          const unsigned ra = q % (unsigned)R, nk = (unsigned)tnk;
          const float wv = tapeW[(size_t)(ra % nk) * (CO * HO * WO) + o];
          t_[r] = ra < nk ? wv : -wv;
        } else {
          t_[r] = tape[(size_t)o * ldq + q];
        }
        if constexpr (ZOUT) {
          const long pi = (long)b * pstride + o;
          l_[r] = a_lo[pi];
          u_[r] = a_up[pi];
          b_[r] = b_up[pi];
        }
      }
    }
  };
  // prologue: the padding columns of every slot are zero for good; the input rows of output
  // row 0, S at a time
  for (int e = threadIdx.x; e < NSLOT * CI * XW * 4; e += 256) {
    const int xr = (e / 4) % XW;
    if (xr < P || xr >= P + WI) *reinterpret_cast<float4v*>(ring + 4 * e) = float4v{0.f, 0.f, 0.f, 0.f};
  }
  for (int yb = y_lo * S - P; yb < y_lo * S + K - P; yb += S) {
    fetch_rows(yb);
    park_rows(yb);
  }
  __syncthreads();
  auto pos_of = [&](int y, int k) { return y * WO + wave / NMT + k * PSTEP; };
  load_ep(pos_of(y_lo, 0), et, el, eu, eb);
  for (int y = y_lo; y < y_hi; ++y) {
    const int ynew = y * S - P + K;  // first input row output row y + 1 adds
    if (y + 1 < y_hi) fetch_rows(ynew);
    int sb[K];  // ring offsets of the K input rows of output row y (uniform)
#pragma unroll
    for (int ky = 0; ky < K; ++ky) sb[ky] = slot_of(y * S - P + ky) * ROWF;
#pragma unroll 1
    for (int k = 0; k < IPW; ++k) {
      const int pos = pos_of(y, k);
      const bool has_next = k + 1 < IPW || y + 1 < y_hi;
      float nt[4], nl[NE], nu[NE], nb[NE];
      if (has_next) load_ep(k + 1 < IPW ? pos_of(y, k + 1) : pos_of(y + 1, 0), nt, nl, nu, nb);
      // this lane's ring column (x*S - P + kx, kx = lane group) plus P; a group kx >= K reads
      // a finite value that meets a zero weight
      const float* col = ring + ((pos - y * WO) * S + g) * 16 + n;
      float4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const float bv = col[sb[ks % K] + (ks / K) * XW * 16];
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(wreg[ks], bv, d, 0, 0, 0);
      }
    if (part) {
      // adjoint terms of the 4 outputs of this lane (rows without weight give exactly 0),
      // summed over each group of 8 rows: w max(A~,0) G, w min(A~,0) G, w min(A~,0)
      float4v sa, da, db;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = mt * 16 + 4 * g + r;
        const float gv = d[r] + (co < CO ? t.b[co] : 0.f);
        const bool on = fz && co < CO;
        const float tp = fmaxf(et[r], 0.f), tn = fminf(et[r], 0.f);
        sa[r] = on ? (wq * tp) * gv : 0.f;
        da[r] = on ? (wq * tn) * gv : 0.f;
        db[r] = on ? wq * tn : 0.f;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sa[r] = sum8(sa[r]);
        da[r] = sum8(da[r]);
        db[r] = sum8(db[r]);
      }
      if ((n & 7) == 0 && mt * 16 + 4 * g < CO) {
        // [group][term][pos][co]: the 4 channels of this lane are contiguous
        const size_t grp = q0 / 8 + (n >> 3);
        float* dst = part + grp * 3 * (NPOS * CO) + (size_t)pos * CO + mt * 16 + 4 * g;
        *reinterpret_cast<float4v*>(dst) = sa;
        *reinterpret_cast<float4v*>(dst + NPOS * CO) = da;
        *reinterpret_cast<float4v*>(dst + 2 * NPOS * CO) = db;
      }
    }
    if (qok && wq != 0.f && (ZOUT || !part)) {
      const int y = pos / WO, x = pos - y * WO;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = mt * 16 + 4 * g + r;
        if (co >= CO) continue;
        const float gv = d[r] + t.b[co];
        const unsigned o = ((unsigned)co * HO + y) * WO + x;
        const size_t idx = (size_t)o * ldq + q;
        if (!part) G[idx] = gv;
        if constexpr (ZOUT) {  // both lines, then a select (no branch)
          const float zl = el[r] * gv, zu = fmaf(eu[r], gv, eb[r]);
          zout[idx] = et[r] >= 0.f ? zl : zu;
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) et[r] = nt[r];
#pragma unroll
    for (int r = 0; r < NE; ++r) {
      el[r] = nl[r];
      eu[r] = nu[r];
      eb[r] = nb[r];
    }
    }  // positions of row y
    if (y + 1 < y_hi) {
      if constexpr (TWO_BAR) __syncthreads();  // the slots ynew takes are free
      park_rows(ynew);
      __syncthreads();
    }
  }
}

// Adjoint accumulation for ReLU layer m: one wave per (sub-domain, neuron) sums over the rows of
// the pass, w * max(A~,0) G (-> alpha), w * min(A~,0) G (-> upper slope) and w * min(A~,0)
// (-> upper intercept), and for unstable neurons turns the last two into adjoints of l and u
// through a_up = u/(u-l), b_up = -u l/(u-l).  Deterministic: fixed lane order and tree.
__global__ void __launch_bounds__(kBlock)
    k_grad_reduce(long nb, long nm, long R, long ldq, const float* __restrict__ w,
                  const float* __restrict__ tape, const float* __restrict__ G,
                  const int8_t* __restrict__ code, const float* __restrict__ l,
                  const float* __restrict__ u, long n_relu, float* __restrict__ ga,
                  float* __restrict__ gl, float* __restrict__ gu) {
  long pair = blockIdx.x * (long)(blockDim.x / 64) + threadIdx.x / 64;
  int lane = threadIdx.x % 64;
  if (pair >= nb * nm) return;  // uniform per wave
  long b = pair / nm, j = pair % nm;
  float sa = 0.f, da = 0.f, db = 0.f;
  for (long r = lane; r < R; r += 64) {
    long q = b * R + r;
    float wr = w[q];
    if (wr == 0.f) continue;
    float tv = tape[j * ldq + q], g = G[j * ldq + q];
    float tp = fmaxf(tv, 0.f), tn = fminf(tv, 0.f);
    sa = fmaf(wr * tp, g, sa);
    da = fmaf(wr * tn, g, da);
    db = fmaf(wr, tn, db);
  }
  for (int o = 32; o >= 1; o >>= 1) {
    sa += __shfl_xor(sa, o, 64);
    da += __shfl_xor(da, o, 64);
    db += __shfl_xor(db, o, 64);
  }
  if (lane != 0) return;
  long p = b * n_relu + j;
  if (code[p] != 5) return;
  float lj = l[p], uj = u[p], d = uj - lj, d2 = d * d;
  ga[p] += sa;
  gl[p] += (da * uj - db * uj * uj) / d2;
  gu[p] += (-da * lj + db * lj * lj) / d2;
}

// The same accumulation when the pass has few rows per sub-domain (R <= 64, e.g. the spec rows
// of the final pass).  The tape and G are [neuron][ldq] with a sub-domain's rows contiguous, so a
// block takes 64 consecutive neurons and SPW = min(floor(64 / R), 16) consecutive sub-domains:
// for each neuron, lane l of a wave reads row q0 + l of the window (coalesced along q), forms
// the row's three terms, and lane s < SPW then sums the R terms of sub-domain b0 + s in row
// order from the wave's LDS scratch.  The block's results are written out with the neurons fastest.  Rows
// with weight 0 contribute nothing and are not read (their G may never have been written).
__global__ void __launch_bounds__(256)
    k_grad_reduce_seg(long nb, long nm, long R, long ldq, const float* __restrict__ w,
                      const float* __restrict__ tape, const float* __restrict__ G,
                      const int8_t* __restrict__ code, const float* __restrict__ l,
                      const float* __restrict__ u, long n_relu, float* __restrict__ ga,
                      float* __restrict__ gl, float* __restrict__ gu) {
  __shared__ float scr[4][3][64];  // per wave: the window's row terms
  __shared__ float res[3][16][65];  // [term][sub-domain slot][neuron] (+1: no bank conflicts)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int SPW = (int)(R >= 4 ? 64 / R : 16), QW = SPW * (int)R;
  const long njt = (nm + 63) / 64;
  const long j0 = (long)(blockIdx.x % njt) * 64;
  const long b0 = (long)(blockIdx.x / njt) * SPW;
  const long q = b0 * R + lane;
  const bool qok = lane < QW && b0 + lane / R < nb;
  const float wq = qok ? w[q] : 0.f;
  // the lane's row's neuron j is unstable in its sub-domain: only those rows' terms are used, so
  // only those rows are read (the codes of the wave's 16 neurons, first)
  bool un[16];
  {
    const long bq = qok ? b0 + lane / R : b0;
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
      const long j = min(j0 + wave * 16 + jj, nm - 1);
      un[jj] = code[bq * n_relu + j] == 5;
    }
  }
#pragma unroll
  for (int jj = 0; jj < 16; ++jj) {
    const int jl = wave * 16 + jj;
    const long j = j0 + jl;
    float ca = 0.f, cd = 0.f, cb = 0.f;
    if (j < nm && wq != 0.f && un[jj]) {
      const float tv = tape[j * ldq + q], g = G[j * ldq + q];
      const float tp = fmaxf(tv, 0.f), tn = fminf(tv, 0.f);
      ca = (wq * tp) * g;
      cd = (wq * tn) * g;
      cb = wq * tn;
    }
    scr[wave][0][lane] = ca;
    scr[wave][1][lane] = cd;
    scr[wave][2][lane] = cb;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the wave's LDS writes are done
    if (lane < SPW) {
      float sa = 0.f, da = 0.f, db = 0.f;
      for (int r = 0; r < (int)R; ++r) {
        sa += scr[wave][0][lane * R + r];
        da += scr[wave][1][lane * R + r];
        db += scr[wave][2][lane * R + r];
      }
      res[0][lane][jl] = sa;
      res[1][lane][jl] = da;
      res[2][lane][jl] = db;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // scr read before the next writes
  }
  __syncthreads();
  for (int e = threadIdx.x; e < SPW * 64; e += 256) {
    const int sl = e >> 6, jl = e & 63;
    const long b = b0 + sl, j = j0 + jl;
    if (b >= nb || j >= nm) continue;
    const long p = b * n_relu + j;
    if (code[p] != 5) continue;
    const float sa = res[0][sl][jl], da = res[1][sl][jl], db = res[2][sl][jl];
    const float lj = l[p], uj = u[p], d = uj - lj, d2 = d * d;
    ga[p] += sa;
    gl[p] += (da * uj - db * uj * uj) / d2;
    gu[p] += (-da * lj + db * lj * lj) / d2;
  }
}

// Projected Adam ascent step (bias-corrected), alpha clipped to [0, 1].
__global__ void __launch_bounds__(kBlock) k_adam(long n, float* __restrict__ alpha,
                                                 float* __restrict__ m, float* __restrict__ v,
                                                 const float* __restrict__ g, float lr,
                                                 float b1, float b2, float eps, float c1,
                                                 float c2) {
  long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i >= n) return;
  float gi = g[i];
  float mi = b1 * m[i] + (1.f - b1) * gi;
  float vi = b2 * v[i] + (1.f - b2) * gi * gi;
  m[i] = mi;
  v[i] = vi;
  float a = alpha[i] + lr * (mi / c1) / (sqrtf(vi / c2) + eps);
  alpha[i] = fminf(fmaxf(a, 0.f), 1.f);
}

// Fresh optimiser state: alpha = the upper slope u/(u-l) of each unstable neuron of a heuristic
// pass (1 for l >= 0, 0 otherwise), Adam moments zero.
__global__ void __launch_bounds__(kBlock) k_alpha_init(long n, const float* __restrict__ l,
                                                       const float* __restrict__ u,
                                                       float* __restrict__ alpha,
                                                       float* __restrict__ m,
                                                       float* __restrict__ v) {
  long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float li = l[i], ui = u[i];
  alpha[i] = (li < 0.f && ui > 0.f) ? ui / (ui - li) : (li >= 0.f ? 1.f : 0.f);
  m[i] = 0.f;
  v[i] = 0.f;
}

// Best bound so far (elementwise max over iterates) and optional trace copy.
__global__ void __launch_bounds__(kBlock) k_best(long n, const float* __restrict__ lb,
                                                 float* __restrict__ best,
                                                 float* __restrict__ trace, int first) {
  long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i >= n) return;
  float v = lb[i];
  best[i] = first ? v : fmaxf(best[i], v);
  if (trace) trace[i] = v;
}

__global__ void __launch_bounds__(kBlock) k_zero(long n, float* __restrict__ p) {
  long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

// Three 16-byte-aligned arrays of n floats cleared in one launch, four floats per store.
__global__ void __launch_bounds__(kBlock)
    k_zero3(long n, float* __restrict__ a, float* __restrict__ b, float* __restrict__ c) {
  const long i = (blockIdx.x * (long)blockDim.x + threadIdx.x) * 4;
  if (i + 4 <= n) {
    const float4v z = {0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<float4v*>(a + i) = z;
    *reinterpret_cast<float4v*>(b + i) = z;
    *reinterpret_cast<float4v*>(c + i) = z;
  } else {
    for (long k = i; k < n; ++k) a[k] = b[k] = c[k] = 0.f;
  }
}

// Spec rows of an upper bound (Eq. 8: max_x U = -min_x of the lower function of -C): out holds
// [C; -C] (both = 1) or -C alone, [rows][nL].
__global__ void __launch_bounds__(kBlock) k_spec_pm(long n, const float* __restrict__ C,
                                                    float* __restrict__ out, int both) {
  long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i >= n) return;
  if (both) {
    out[i] = C[i];
    out[n + i] = -C[i];
  } else {
    out[i] = -C[i];
  }
}

// Bounds of the rows [C; -C] of nb sub-domains ([nb][2S]) into lb = the C rows and
// ub = -(the -C rows), [nb][S] each.
__global__ void __launch_bounds__(kBlock) k_split_ul(long nb, long S, const float* __restrict__ lb2,
                                                     float* __restrict__ lb, float* __restrict__ ub) {
  long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i >= nb * S) return;
  const long b = i / S, s_ = i % S;
  lb[i] = lb2[b * 2 * S + s_];
  ub[i] = -lb2[b * 2 * S + S + s_];
}

__global__ void __launch_bounds__(kBlock) k_negate(long n, float* __restrict__ p) {
  long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i < n) p[i] = -p[i];
}


// ---------------------------------------------------------------------------------------------
// Branch and bound (Algorithm 1 without the LP fallback)
// ---------------------------------------------------------------------------------------------
// The set P of unverified sub-domains lives on the device as a store of records: split mask
// [n_relu] int8, slopes alpha [n_relu], f_lo, f_hi and the neuron to split next.  The batch of
// children of an iteration has the same layout.

// Branching stand-in (BaBSR's score is not given in the paper): the unstable, unsplit neuron
// with the largest intercept -l u / (u - l) of its upper relaxation line (Eq. 5) under the
// sub-domain's own bounds; the lowest flat index on ties; -1 when none is left.  One block per
// sub-domain.
__global__ void __launch_bounds__(kBlock)
    k_bab_branch(long n_relu, const float* __restrict__ l, const float* __restrict__ u,
                 const int8_t* __restrict__ code, int* __restrict__ branch) {
  __shared__ float bs[kBlock];
  __shared__ int bj[kBlock];
  const long b = blockIdx.x;
  float best = -INFINITY;
  int jb = -1;
  for (long j = threadIdx.x; j < n_relu; j += kBlock) {
    const long p = b * n_relu + j;
    if (code[p] != 5) continue;
    const float lj = l[p], uj = u[p];
    const float sc = -(lj * uj) / (uj - lj);
    if (sc > best) {  // j increases within a thread: the first maximum is kept
      best = sc;
      jb = (int)j;
    }
  }
  bs[threadIdx.x] = best;
  bj[threadIdx.x] = jb;
  __syncthreads();
  for (int o = kBlock / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      const float s2 = bs[threadIdx.x + o];
      const int j2 = bj[threadIdx.x + o];
      if (j2 >= 0 && (bj[threadIdx.x] < 0 || s2 > bs[threadIdx.x] ||
                      (s2 == bs[threadIdx.x] && j2 < bj[threadIdx.x]))) {
        bs[threadIdx.x] = s2;
        bj[threadIdx.x] = j2;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) branch[b] = bj[0];
}

// Summary of P read by the host after every iteration.
struct BabSummary {
  int count;     // |P|
  int stuck;     // a sub-domain among the next batch has no neuron left to split
  float f_lo;    // min over P of the lower bounds (Algorithm 1, line 9)
  float f_hi;    // min over P of the upper bounds (line 10)
  float leaf_lo; // min lower bound of the verified sub-domains dropped so far
  float leaf_hi; // min upper bound of those
  int pad[2];
};

__device__ __forceinline__ unsigned int ordered_bits(float f) {
  const unsigned int b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// batch_pick_out (line 5): one block sorts the N = sum->count records of P by (f_lo, slot)
// ascending with a bitonic network in LDS (N rounded up to a power of two, at most the LDS the
// launch reserved) and writes the order to perm; then fills the summary (stuck looks at the
// first min(batch, N) records).
__global__ void __launch_bounds__(1024)
    k_bab_sort(int batch, const float* __restrict__ lo, const float* __restrict__ hi,
               const int* __restrict__ branch, int* __restrict__ perm,
               BabSummary* __restrict__ sum) {
  extern __shared__ unsigned long long keys[];
  __shared__ float red[1024];
  __shared__ int stk[1024];
  const int tid = threadIdx.x;
  const int N = sum->count;
  int npad = 1;
  while (npad < N) npad <<= 1;
  for (int i = tid; i < npad; i += 1024)
    keys[i] = i < N ? ((unsigned long long)ordered_bits(lo[i]) << 32) | (unsigned)i
                    : ~0ull;
  __syncthreads();
  for (int k = 2; k <= npad; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < npad; i += 1024) {
        const int ix = i ^ j;
        if (ix > i) {
          const unsigned long long a = keys[i], c = keys[ix];
          const bool up = (i & k) == 0;
          if ((a > c) == up) {
            keys[i] = c;
            keys[ix] = a;
          }
        }
      }
      __syncthreads();
    }
  float mh = INFINITY;
  int st = 0;
  const int kb = min(batch, N);
  for (int i = tid; i < N; i += 1024) {
    const int slot = (int)(keys[i] & 0xffffffffu);
    perm[i] = slot;
    mh = fminf(mh, hi[slot]);
    if (i < kb && branch[slot] < 0) st = 1;
  }
  red[tid] = mh;
  stk[tid] = st;
  __syncthreads();
  for (int o = 512; o > 0; o >>= 1) {
    if (tid < o) {
      red[tid] = fminf(red[tid], red[tid + o]);
      stk[tid] |= stk[tid + o];
    }
    __syncthreads();
  }
  if (tid == 0) {
    sum->count = N;
    sum->stuck = stk[0];
    sum->f_lo = N > 0 ? lo[(int)(keys[0] & 0xffffffffu)] : INFINITY;
    sum->f_hi = red[0];
  }
}

// batch_split (line 6): child 2i of the i-th picked record forces its branching neuron active
// (+1), child 2i + 1 inactive (-1); both start from the parent's slopes.
__global__ void __launch_bounds__(kBlock)
    k_bab_children(long k, long n_relu, const int* __restrict__ perm,
                   const int8_t* __restrict__ smask, const float* __restrict__ salpha,
                   const int* __restrict__ sbranch, int8_t* __restrict__ cmask,
                   float* __restrict__ calpha) {
  const long idx = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (idx >= 2 * k * n_relu) return;
  const long c = idx / n_relu, j = idx % n_relu;
  const long par = perm[c >> 1];
  const int8_t v = smask[par * n_relu + j];
  cmask[idx] = j == sbranch[par] ? (int8_t)((c & 1) ? -1 : 1) : v;
  if (calpha) calpha[idx] = salpha[par * n_relu + j];
}

// The records of P that were not picked (perm[k..N)) into the other store buffer, in order.
__global__ void __launch_bounds__(kBlock)
    k_bab_gather(long nrest, long k, long n_relu, const int* __restrict__ perm,
                 const int8_t* __restrict__ smask, const float* __restrict__ salpha,
                 const float* __restrict__ slo, const float* __restrict__ shi,
                 const int* __restrict__ sbranch, int8_t* __restrict__ dmask,
                 float* __restrict__ dalpha, float* __restrict__ dlo, float* __restrict__ dhi,
                 int* __restrict__ dbranch) {
  const long idx = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (idx >= nrest * n_relu) return;
  const long r = idx / n_relu, j = idx % n_relu;
  const long src = perm[k + r];
  dmask[idx] = smask[src * n_relu + j];
  if (dalpha) dalpha[idx] = salpha[src * n_relu + j];
  if (j == 0) {
    dlo[r] = slo[src];
    dhi[r] = shi[src];
    dbranch[r] = sbranch[src];
  }
}

// Domain_Filter (line 8): children with f_lo >= 0 are verified and dropped (their bounds kept
// in the summary's leaf minima); the others get consecutive slots from N0 on, in child order.
// One block; nc <= 2048.
__global__ void __launch_bounds__(1024)
    k_bab_filter(int nc, int N0, const float* __restrict__ clo, const float* __restrict__ chi,
                 int* __restrict__ dst, BabSummary* __restrict__ sum) {
  __shared__ int cnt[1024];
  __shared__ float rl[1024], rh[1024];
  const int tid = threadIdx.x;
  const int c0 = 2 * tid, c1 = 2 * tid + 1;
  const bool k0 = c0 < nc && !(clo[c0] >= 0.f), k1 = c1 < nc && !(clo[c1] >= 0.f);
  float ll = INFINITY, lh = INFINITY;
  if (c0 < nc && !k0) { ll = clo[c0]; lh = chi[c0]; }
  if (c1 < nc && !k1) { ll = fminf(ll, clo[c1]); lh = fminf(lh, chi[c1]); }
  cnt[tid] = (int)k0 + (int)k1;
  rl[tid] = ll;
  rh[tid] = lh;
  __syncthreads();
  // inclusive scan (Hillis-Steele) of the kept counts; minima of the dropped bounds
  for (int o = 1; o < 1024; o <<= 1) {
    const int v = tid >= o ? cnt[tid - o] : 0;
    __syncthreads();
    cnt[tid] += v;
    __syncthreads();
  }
  for (int o = 512; o > 0; o >>= 1) {
    if (tid < o) {
      rl[tid] = fminf(rl[tid], rl[tid + o]);
      rh[tid] = fminf(rh[tid], rh[tid + o]);
    }
    __syncthreads();
  }
  const int before = cnt[tid] - (int)k0 - (int)k1;
  if (c0 < nc) dst[c0] = k0 ? N0 + before : -1;
  if (c1 < nc) dst[c1] = k1 ? N0 + before + (int)k0 : -1;
  if (tid == 0) {
    sum->leaf_lo = fminf(sum->leaf_lo, rl[0]);
    sum->leaf_hi = fminf(sum->leaf_hi, rh[0]);
    sum->count = N0 + cnt[1023];
  }
}

// Kept children into their slots of P.
__global__ void __launch_bounds__(kBlock)
    k_bab_insert(long nc, long n_relu, const int* __restrict__ dst,
                 const int8_t* __restrict__ cmask, const float* __restrict__ calpha,
                 const float* __restrict__ clo, const float* __restrict__ chi,
                 const int* __restrict__ cbranch, int8_t* __restrict__ smask,
                 float* __restrict__ salpha, float* __restrict__ slo, float* __restrict__ shi,
                 int* __restrict__ sbranch) {
  const long idx = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (idx >= nc * n_relu) return;
  const long c = idx / n_relu, j = idx % n_relu;
  const int d = dst[c];
  if (d < 0) return;
  smask[(long)d * n_relu + j] = cmask[idx];
  if (salpha) salpha[(long)d * n_relu + j] = calpha[idx];
  if (j == 0) {
    slo[d] = clo[c];
    shi[d] = chi[c];
    sbranch[d] = cbranch[c];
  }
}

__global__ void __launch_bounds__(kBlock) k_fill_i8(long n, int8_t* __restrict__ p, int v) {
  const long i = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if (i < n) p[i] = (int8_t)v;
}

__global__ void k_bab_summary_init(BabSummary* sum) {
  sum->count = 0;
  sum->stuck = 0;
  sum->f_lo = INFINITY;
  sum->f_hi = INFINITY;
  sum->leaf_lo = INFINITY;
  sum->leaf_hi = INFINITY;
}

// ---------------------------------------------------------------------------------------------
// Input check (LIRPA_VALIDATE=1)
// ---------------------------------------------------------------------------------------------
__global__ void __launch_bounds__(kBlock)
    k_check_inputs(long n_split, const int8_t* __restrict__ split, long n_alpha,
                   const float* __restrict__ alpha, long n_x0, const float* __restrict__ x0,
                   long n_C, const float* __restrict__ C) {
  const long stride = (long)gridDim.x * blockDim.x;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n_split; i += stride) {
    const int v = split[i];
    if (v < -1 || v > 1) g_check[0] = 1u;
  }
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n_alpha; i += stride) {
    const float a = alpha[i];
    if (!(a >= 0.f && a <= 1.f)) g_check[1] = 1u;
  }
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n_x0; i += stride)
    if (!isfinite(x0[i])) g_check[2] = 1u;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n_C; i += stride)
    if (!isfinite(C[i])) g_check[3] = 1u;
}

// ---------------------------------------------------------------------------------------------
// Workspace plan
// ---------------------------------------------------------------------------------------------
struct Plan {
  long Bc = 0;
  int mode = 0;
  size_t off_l = 0, off_u = 0, off_alo = 0, off_aup = 0, off_bup = 0, off_code = 0;
  size_t off_l1u1 = 0, off_slab0 = 0, off_slab1 = 0, off_beta = 0, total = 0;
  size_t off_wsp = 0;  // C W_L [S][n_{L-1}], then C b_L [S] (L >= 2, T_L fully connected)
  size_t off_bz = 0;  // per-neuron bias of every ReLU layer (padded layout, segment m at poff[m])
  size_t off_z1 = 0;  // its layer-1 segment: W1 x0 + b1
  long slab_floats = 0, qp_max = 0;
  // mode 1 (gradient): tape[k][m] holds, for pass k, the coefficients over g^(m) before their
  // relaxation (m >= 1) and over x (m = 0), [n_m][qp_k]; adjoints; row weights; forward slabs.
  size_t off_tape[kMaxLayers + 1][kMaxLayers + 1] = {};
  size_t off_wT[kMaxLayers + 1] = {};  // transposed FC weights of layers 2..L-1 (0 = none)
  size_t off_ga = 0, off_gl = 0, off_gu = 0, off_w = 0, off_za = 0, off_zb = 0, off_G = 0;
  size_t off_lbt = 0, off_grad = 0, off_p2part = 0, off_p2flag = 0;
  // adjoint partial sums of the fused witness forward, [Qp/8][3][n_m], and a flag per group of
  // 8 rows (whether any row of the group carries weight)
  size_t off_gpart = 0, off_gflag = 0;
  size_t off_gpart2 = 0;  // layer-2 partial sums of the fused two-layer witness forward
  size_t off_w2t = 0;     // its copy of T_2's weights with the tap indices exchanged
  size_t off_w3c = 0;     // and of T_3's weights with the input index channel-last
  size_t off_kidx1 = 0, off_list1 = 0, off_cnt1 = 0;  // its unstable layer-1 neurons' ranks
  size_t off_kidx2 = 0, off_list2 = 0, off_cnt2 = 0;  // and layer-2 neurons'
  size_t off_psel = 0;  // its position pairs of layer-2 tiles per sub-domain
  long fwd_floats = 0;
  // lower and upper bounds in one call: the spec rows [C; -C] (or -C alone) and, for the bound,
  // the [Bc][2S] bounds of those rows before they are split into lb and ub
  size_t off_spec = 0, off_lb2 = 0;
};

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Kernel for the receptive-field pass 2, or null when the shapes do not qualify.
using Pass2Kernel = void (*)(DLayer, DLayer, long, const float*, const float*, const float*, long,
                             const float*, float, float*, float*, long, long, const int8_t*,
                             const float*, float*, float*, float*, int8_t*, const float*,
                             const float*);
// Windows per block of the receptive-field pass 2 (along x2): 8 when the map width allows it
// (fewer blocks, each set-up shared by more windows), else 4.
int p2_xw(const lirpa_net* net) { return net->T[1].out_w % 8 == 0 ? 8 : 4; }

template <int XW>
Pass2Kernel pass2_kernel_xw(const lirpa_layer& t1, const lirpa_layer& t2) {
  if (t1.k == 4 && t1.stride == 2 && t1.pad == 1 && t1.in_c == 3) {
    if (t2.k == 4 && t1.out_c == 8) return k_pass2_window<4, 2, 1, 4, 8, 3, XW>;
    if (t2.k == 4 && t1.out_c == 16) return k_pass2_window<4, 2, 1, 4, 16, 3, XW>;
    if (t2.k == 3 && t1.out_c == 8) return k_pass2_window<4, 2, 1, 3, 8, 3, XW>;
  }
  return nullptr;
}

Pass2Kernel pass2_kernel_for(const lirpa_net* net, int* nw) {
  if (net->L < 3) return nullptr;
  if (net->T[1].out_w % 4) return nullptr;
  const lirpa_layer &t1 = net->T[0], &t2 = net->T[1];
  if (t1.kind != LIRPA_CONV2D || t2.kind != LIRPA_CONV2D) return nullptr;
  if ((t2.out_c % 16 && t2.out_c != 8) || t1.in_c > 8) return nullptr;
  *nw = t1.in_c;
  return p2_xw(net) == 8 ? pass2_kernel_xw<8>(t1, t2) : pass2_kernel_xw<4>(t1, t2);
}

using Pass2GradKernel = void (*)(DLayer, DLayer, const float*, const float*, long, float,
                                 const float*, const float*, const int8_t*, long, long,
                                 const float*, float*, unsigned char*);
Pass2GradKernel pass2_grad_kernel_for(const lirpa_net* net) {
  int nw = 0;
  if (!pass2_kernel_for(net, &nw)) return nullptr;
  const lirpa_layer &t1 = net->T[0], &t2 = net->T[1];
  // windows per block: those of k_pass2_window
  if (p2_xw(net) == 8) {
    if (t2.k == 4 && t1.out_c == 8) return k_pass2_window_grad<4, 2, 1, 4, 8, 3, 8>;
    if (t2.k == 4 && t1.out_c == 16) return k_pass2_window_grad<4, 2, 1, 4, 16, 3, 8>;
    if (t2.k == 3 && t1.out_c == 8) return k_pass2_window_grad<4, 2, 1, 3, 8, 3, 8>;
  } else {
    if (t2.k == 4 && t1.out_c == 8) return k_pass2_window_grad<4, 2, 1, 4, 8, 3, 4>;
    if (t2.k == 4 && t1.out_c == 16) return k_pass2_window_grad<4, 2, 1, 4, 16, 3, 4>;
    if (t2.k == 3 && t1.out_c == 8) return k_pass2_window_grad<4, 2, 1, 3, 8, 3, 4>;
  }
  return nullptr;
}

long pass2_blocks(const lirpa_net* net, long nb) {
  const lirpa_layer& t2 = net->T[1];
  return nb * p2_groups(t2.out_c) * t2.out_h * t2.out_w;
}

// Whether bound mode (no gradient tape) runs pass k, 2 <= k < L, in one kernel that keeps the
// pass's coefficients on chip: such a pass needs no bound-matrix slab.
bool pass_on_chip(const lirpa_net* net, int k, long Bc);

// The fused two-layer witness forward of pass 3 (k_fwd_conv12) for a net whose T_1 is
// Conv(3 -> C1, k4 s2 p1, 32x32), T_2 Conv(C1 -> C2, k4 s2 p1, 16x16) and T_3 Linear, with
// (C1, C2) = (8, 16) or (16, 32); null otherwise.
using Fwd12Kernel = void (*)(DLayer, DLayer, const int8_t*, unsigned, unsigned, unsigned,
                             const float*, const float*, float, const float*, const float*,
                             const float*, const float*, unsigned, const float*, unsigned,
                             unsigned, const unsigned*, const int*, const int*,
                             const float*, float*, float*, unsigned char*);
Fwd12Kernel fwd12_for(const lirpa_net* net) {
  if (net->L < 4 || net->T[2].kind != LIRPA_LINEAR) return nullptr;
  const lirpa_layer &a = net->T[0], &t = net->T[1];
  if (a.kind != LIRPA_CONV2D || t.kind != LIRPA_CONV2D) return nullptr;
  const bool ga = a.k == 4 && a.stride == 2 && a.pad == 1 && a.in_c == 3 && a.in_h == 32 &&
                  a.in_w == 32 && a.out_h == 16 && a.out_w == 16;
  const bool gt = t.k == 4 && t.stride == 2 && t.pad == 1 && t.in_h == 16 && t.in_w == 16 &&
                  t.out_h == 8 && t.out_w == 8;
  if (!ga || !gt) return nullptr;
  if (a.out_c == 8 && t.out_c == 16) return k_fwd_conv12<8, 16>;
  if (a.out_c == 16 && t.out_c == 32) return k_fwd_conv12<16, 32>;
  return nullptr;
}

Plan make_plan(const lirpa_net* net, long S, long Bc, int mode = 0) {
  Plan p;
  p.Bc = Bc;
  p.mode = mode;
  const int L = net->L;
  long slab = 0, qpmax = round_up(2 * net->n[1], 64);
  int nw_unused = 0;
  const bool win2 = (mode == 0 && pass2_kernel_for(net, &nw_unused) != nullptr) ||
                    (mode == 1 && pass2_grad_kernel_for(net) != nullptr);
  for (int k = 2; k <= L; ++k) {
    long R = (k < L) ? 2 * net->n[k] : S;
    long qp = round_up(Bc * R, 64);
    if (k == 2 && win2 && k < L) continue;
    qpmax = std::max(qpmax, qp);
    if (mode == 0 && k < L && pass_on_chip(net, k, Bc)) continue;
    int mtop = (k < L) ? k - 1 : L;  // slabs hold A over h^(m), m = mtop..1
    for (int m = 1; m <= mtop; ++m) slab = std::max(slab, net->n[m] * qp);
  }
  if (L == 1) {
    long qp = round_up(Bc * S, 64);
    qpmax = std::max(qpmax, qp);
    slab = std::max(slab, net->n[1] * qp);
  }
  p.slab_floats = slab;
  p.qp_max = qpmax;
  size_t o = 0;
  size_t per = (size_t)Bc * (net->n_relu ? net->n_relu : 1);
  size_t perp = (size_t)Bc * (net->pstride ? net->pstride : 4);
  p.off_l = o;    o = align256(o + per * 4);
  p.off_u = o;    o = align256(o + per * 4);
  p.off_alo = o;  o = align256(o + perp * 4);
  p.off_aup = o;  o = align256(o + perp * 4);
  p.off_bup = o;  o = align256(o + perp * 4);
  p.off_code = o; o = align256(o + per);
  p.off_l1u1 = o; o = align256(o + 2 * (size_t)net->n[1] * 4);
  if (net->L >= 2 && net->T[net->L - 1].kind == LIRPA_LINEAR) {
    p.off_wsp = o;
    o = align256(o + (size_t)S * (net->n[net->L - 1] + 1) * 4);
  }
  p.off_bz = o;   o = align256(o + (size_t)std::max<long>(net->pstride, net->n[1]) * 4);
  p.off_z1 = p.off_bz + (size_t)net->poff[1] * 4;
  p.off_beta = o; o = align256(o + (size_t)qpmax * 4);
  p.off_slab0 = o; o = align256(o + (size_t)slab * 4);
  p.off_slab1 = o; o = align256(o + (size_t)slab * 4);
  for (int k = 2; k <= L - 1; ++k)
    if (net->T[k - 1].kind == LIRPA_LINEAR) {
      p.off_wT[k] = o;
      o = align256(o + (size_t)net->n[k] * net->n[k - 1] * 4);
    }
  if (mode == 1) {
    long fwd = 0;
    for (int k = 2; k <= L; ++k) {
      long R = (k < L) ? 2 * net->n[k] : S;
      long qp = round_up(Bc * R, 64);
      if (k == 2 && win2 && k < L) {
        // pass 2 is differentiated window by window: partial sums per block and window neuron
        const lirpa_layer& t2 = net->T[1];
        const int k2 = t2.k;
        p.off_p2part = o;
        o = align256(o + (size_t)pass2_blocks(net, Bc) * net->T[0].out_c * k2 * k2 * 4);
        p.off_p2flag = o;  // one byte per window: has a live row
        o = align256(o + (size_t)pass2_blocks(net, Bc));
        continue;
      }
      for (int m = 0; m <= k - 1; ++m) {
        p.off_tape[k][m] = o;  // over x: signs, one byte per entry
        o = align256(o + (size_t)net->n[m] * qp * (m == 0 ? 1 : 4));
        if (m >= 1) fwd = std::max(fwd, net->n[m] * qp);
      }
    }
    p.fwd_floats = fwd;
    p.off_ga = o; o = align256(o + per * 4);
    p.off_gl = o; o = align256(o + per * 4);
    p.off_gu = o; o = align256(o + per * 4);
    p.off_grad = o; o = align256(o + per * 4);
    p.off_w = o;  o = align256(o + (size_t)qpmax * 4);
    p.off_za = o; o = align256(o + (size_t)fwd * 4);
    p.off_zb = o; o = align256(o + (size_t)fwd * 4);
    p.off_G = o;  o = align256(o + (size_t)fwd * 4);
    p.off_lbt = o; o = align256(o + (size_t)Bc * S * 4);
    long gpart = 0, gflag = 0;
    for (int k = 2; k <= L - 1; ++k) {
      if ((k == 2 && win2) || (2 * net->n[k]) % 8) continue;
      const long qp8 = round_up(Bc * 2 * net->n[k], 64) / 8;
      gflag = std::max(gflag, qp8);
      for (int m = 1; m <= k - 1; ++m) gpart = std::max(gpart, qp8 * 3 * net->n[m]);
    }
    p.off_gpart = o; o = align256(o + (size_t)gpart * 4);
    p.off_gflag = o; o = align256(o + (size_t)gflag);
    if (fwd12_for(net)) {
      // pass 3's layer-2 partial sums, written by the same kernel as its layer-1 sums
      p.off_gpart2 = o;
      o = align256(o + (size_t)(round_up(Bc * 2 * net->n[3], 64) / 8) * 3 * net->n[2] * 4);
      const lirpa_layer& t2 = net->T[1];
      p.off_w2t = o;
      o = align256(o + (size_t)t2.out_c * t2.in_c * t2.k * t2.k * 4);
      p.off_w3c = o;
      o = align256(o + (size_t)net->T[2].out_c * net->T[2].in_c * 4);
      p.off_kidx1 = o;
      o = align256(o + (size_t)Bc * net->n[1] * 4);
      p.off_list1 = o;
      o = align256(o + (size_t)Bc * net->n[1] * 4);
      p.off_cnt1 = o;
      o = align256(o + (size_t)Bc * 4);
      p.off_kidx2 = o;
      o = align256(o + (size_t)Bc * net->n[2] * 4);
      p.off_list2 = o;
      o = align256(o + (size_t)Bc * net->n[2] * 4);
      p.off_cnt2 = o;
      o = align256(o + (size_t)Bc * 4);
      p.off_psel = o;  // k_pair_select's [Bc][4][H2][2] words (H2 = 8)
      o = align256(o + (size_t)Bc * 4 * 8 * 2 * 4);
    }
  }
  p.total = o;
  // kernels address a slab with 32-bit element offsets
  long big = std::max(slab, p.fwd_floats);
  if (mode == 1)
    for (int k = 2; k <= L; ++k) {
      if (k == 2 && win2 && k < L) continue;
      big = std::max(big, net->n[0] * round_up(Bc * ((k < L) ? 2 * net->n[k] : S), 64));
    }
  if (big >= (1L << 31)) p.total = (size_t)-1;
  return p;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

dim3 grid_for(long n) { return dim3((unsigned)((n + kBlock - 1) / kBlock)); }

// One backward stage through layer m (1-based) applied to Q rows held in `in` ([n_m][ldq]).
// Geometries with an MFMA transposed-convolution kernel: (k, stride, pad, out_h, out_w, in_h,
// in_w) of the forward layer.  Other shapes use the per-lane gather kernel.
template <int MODE>
using ConvTKernel = void (*)(DLayer, const float*, unsigned, unsigned, Sink);

// Block size limit per instantiation: 256 threads (one wave per SIMD, so the unified register
// file can hold the 32-wide ring of accumulators) for in_c <= 8, else 512.
// Geometry / channel combinations with an MFMA kernel (k4 s2 p1 from 3 to 8 or 16 channels on
// 32x32, k4 s2 p1 from 8 or 16 to 16 or 32 channels on 16x16, k3 s1 p1 8 to 8 on 16x16);
// everything else uses the per-lane gather kernel.  One wave per channel ci, two
// channels per wave above 8.
template <int MODE, bool TAPE>
ConvTKernel<MODE> convT_mfma_pick(const DLayer& t, int* nwaves) {
  const bool g_s2_32 = t.k == 4 && t.stride == 2 && t.pad == 1 && t.out_h == 16 &&
                       t.out_w == 16 && t.in_h == 32 && t.in_w == 32;
  const bool g_s2_16 = t.k == 4 && t.stride == 2 && t.pad == 1 && t.out_h == 8 && t.out_w == 8 &&
                       t.in_h == 16 && t.in_w == 16;
  const bool g_s1_16 = t.k == 3 && t.stride == 1 && t.pad == 1 && t.out_h == 16 &&
                       t.out_w == 16 && t.in_h == 16 && t.in_w == 16;
  if (g_s2_32 && t.in_c == 3 && t.out_c == 8) {
    *nwaves = 3;
    return k_convT_mfma<4, 2, 1, 16, 16, 32, 32, 8, 1, 3, MODE, TAPE>;
  }
  if (g_s2_32 && t.in_c == 3 && t.out_c == 16) {
    *nwaves = 3;
    return k_convT_mfma<4, 2, 1, 16, 16, 32, 32, 16, 1, 3, MODE, TAPE>;
  }
  if (g_s2_16 && t.in_c == 8 && t.out_c == 16) {
    *nwaves = 8;
    return k_convT_mfma<4, 2, 1, 8, 8, 16, 16, 16, 1, 8, MODE, TAPE>;
  }
  if (g_s2_16 && t.in_c == 8 && t.out_c == 8) {
    *nwaves = 8;
    return k_convT_mfma<4, 2, 1, 8, 8, 16, 16, 8, 1, 8, MODE, TAPE>;
  }
  if (g_s2_16 && t.in_c == 16 && t.out_c == 32) {
    *nwaves = 8;
    return k_convT_mfma<4, 2, 1, 8, 8, 16, 16, 32, 2, 8, MODE, TAPE>;
  }
  if (g_s1_16 && t.in_c == 8 && t.out_c == 8) {
    *nwaves = 8;
    return k_convT_mfma<3, 1, 1, 16, 16, 16, 16, 8, 1, 8, MODE, TAPE>;
  }
  return nullptr;
}

// Geometry / channel combinations with an MFMA kernel (k4 s2 p1 from 3 to 8 or 16 channels on
// 32x32, k4 s2 p1 from 8 or 16 to 16 or 32 channels on 16x16, k3 s1 p1 8 to 8 on 16x16);
// everything else uses the per-lane gather kernel.  One wave per channel ci, two
// channels per wave above 8.
template <int MODE>
ConvTKernel<MODE> convT_mfma_for(const DLayer& t, bool tape, int* nwaves) {
  return tape ? convT_mfma_pick<MODE, true>(t, nwaves) : convT_mfma_pick<MODE, false>(t, nwaves);
}

// Wave-specialised relaxing stage for the 16-wide output geometries; null when not covered.
// fc: the variant that builds its input from the fully connected layer above (bound passes
// only).  *nwaves: matrix + storer waves; *lds: dynamic LDS bytes.
using WsKernel = void (*)(DLayer, const float*, unsigned, unsigned, Sink, FcSrc);
template <int K, int S, int P, int H1, int W1, int H0, int W0, int CO, int CI, int CPW, int NS>
WsKernel convT_ws_inst(bool tape, bool fc, int* nwaves, size_t* lds) {
  *nwaves = CI / CPW + NS;
  *lds = 0;  // all LDS of the kernel is static
  if (fc)
    return tape ? k_convT_relax_ws<K, S, P, H1, W1, H0, W0, CO, CI, CPW, NS, true, true>
                : k_convT_relax_ws<K, S, P, H1, W1, H0, W0, CO, CI, CPW, NS, false, true>;
  return tape ? k_convT_relax_ws<K, S, P, H1, W1, H0, W0, CO, CI, CPW, NS, true, false>
              : k_convT_relax_ws<K, S, P, H1, W1, H0, W0, CO, CI, CPW, NS, false, false>;
}

WsKernel convT_ws_for(const DLayer& t, bool tape, bool fc, int* nwaves, size_t* lds) {
  const bool g_s2_16 = t.k == 4 && t.stride == 2 && t.pad == 1 && t.out_h == 8 && t.out_w == 8 &&
                       t.in_h == 16 && t.in_w == 16;
  const bool g_s1_16 = t.k == 3 && t.stride == 1 && t.pad == 1 && t.out_h == 16 &&
                       t.out_w == 16 && t.in_h == 16 && t.in_w == 16;
  if (g_s2_16 && t.in_c == 8 && t.out_c == 16)
    return fc ? convT_ws_inst<4, 2, 1, 8, 8, 16, 16, 16, 8, 1, 4>(tape, fc, nwaves, lds)
              : convT_ws_inst<4, 2, 1, 8, 8, 16, 16, 16, 8, 2, 4>(tape, fc, nwaves, lds);
  if (g_s2_16 && t.in_c == 8 && t.out_c == 8)
    return convT_ws_inst<4, 2, 1, 8, 8, 16, 16, 8, 8, 1, 4>(tape, fc, nwaves, lds);
  if (g_s2_16 && t.in_c == 16 && t.out_c == 32)
    return convT_ws_inst<4, 2, 1, 8, 8, 16, 16, 32, 16, 2, 4>(tape, fc, nwaves, lds);
  if (g_s1_16 && t.in_c == 8 && t.out_c == 8 && !fc)
    return convT_ws_inst<3, 1, 1, 16, 16, 16, 16, 8, 8, 1, 4>(tape, fc, nwaves, lds);
  return nullptr;
}

template <int MODE>
int launch_stage(const lirpa_net* net, int m, int pass, const float* in, long ldq, long Q,
                 const Sink& s, hipStream_t st) {
  DLayer t = dlayer(net->T[m - 1]);
  const char* sfx = MODE == MODE_SLAB ? "_relax" : "_bound";
  const unsigned nblk32 = (unsigned)((Q + 31) / 32);
  if (t.kind == LIRPA_LINEAR) {
    if (t.out_c <= 448) {
      // few row tiles (a final pass): 16 waves per block, so that each wave carries fewer
      // output tiles in sequence
      const bool wide = nblk32 <= 256;
      const int nwv = wide ? 16 : 8;
      size_t lds = ((size_t)t.out_c * 32 + (size_t)nwv * 3 * 32) * sizeof(float);
      return launch_k(tag((std::string("fcT") + sfx).c_str(), m, pass), st, [&] {
        if (wide)
          hipLaunchKernelGGL((k_fcT_mfma<MODE, 16>), dim3(nblk32), dim3(1024), lds, st, t, in,
                             ldq, Q, s);
        else
          hipLaunchKernelGGL((k_fcT_mfma<MODE, 8>), dim3(nblk32), dim3(512), lds, st, t, in, ldq,
                             Q, s);
      });
    }
    return launch_k(tag((std::string("fcT_lane") + sfx).c_str(), m, pass), st, [&] {
      hipLaunchKernelGGL(k_fcT<MODE>, grid_for(Q), dim3(kBlock), 0, st, t, in, ldq, Q, s);
    });
  }
  int nw = 0;
  if constexpr (MODE == MODE_SLAB) {
    if (s.R >= 16) {
      int nwt = 0;
      size_t lds = 0;
      if (WsKernel kern = convT_ws_for(t, s.tape != nullptr, false, &nwt, &lds)) {
        const unsigned nblk16 = (unsigned)round_up((Q + 15) / 16, 16);
        return launch_k(tag("convT_relax", m, pass), st, [&] {
          hipLaunchKernelGGL(kern, dim3(nblk16), dim3(64 * nwt), lds, st, t, in, (unsigned)ldq,
                             (unsigned)Q, s, FcSrc{});
        });
      }
    }
  }
  const bool tape = MODE == MODE_SLAB ? s.tape != nullptr : s.tsign != nullptr;
  if (ConvTKernel<MODE> kern = convT_mfma_for<MODE>(t, tape, &nw)) {
    const unsigned nblk16 = (unsigned)round_up((Q + 15) / 16, 16);
    const size_t cs = (size_t)t.out_w * 16 + (80 - (t.out_w * 16) % 64) % 64;
    // x0 is staged in LDS only when the linear term is not folded into the layer-1 bias
    size_t lds = (2 * (size_t)t.out_c * cs + (size_t)nw * 3 * 16 +
                  (MODE == MODE_BOUND && s.x0 ? (size_t)t.in_c * t.in_h * t.in_w : 0)) *
                 sizeof(float);
    return launch_k(tag((std::string("convT") + sfx).c_str(), m, pass), st, [&] {
      hipLaunchKernelGGL(kern, dim3(nblk16), dim3(64 * nw), lds, st, t, in, (unsigned)ldq,
                         (unsigned)Q, s);
    });
  }
  return launch_k(tag((std::string("convT_lane") + sfx).c_str(), m, pass), st, [&] {
    hipLaunchKernelGGL(k_convT<MODE>, grid_for(Q), dim3(kBlock), 0, st, t, in, ldq, Q, s);
  });
}

struct Chunk {
  const lirpa_net* net;
  const Plan* p;
  void* ws;
  const float* x0;
  float eps;
  long S;
  long nb;             // sub-domains in this chunk
  float* L;            // l rows of the chunk, stride n_relu
  float* U;
  const int8_t* split; // chunk's first row or null
  const float* alpha;
  hipStream_t st;
  bool tape = false;   // record the gradient tape (mode-1 plan)
  const float* lp = nullptr;  // the parent sub-domains' l, u (chunk's first row) or null
  const float* up = nullptr;
};

// Sink that relaxes onto ReLU layer m and stores into `out`.
Sink slab_sink(const Chunk& c, int m, float* out, long ldq, long R) {
  const lirpa_net* net = c.net;
  const lirpa_layer& t = net->T[m - 1];
  Sink s{};
  s.out = out;
  s.ldq = ldq;
  s.a_lo = at<float>(c.ws, c.p->off_alo) + net->poff[m];
  s.a_up = at<float>(c.ws, c.p->off_aup) + net->poff[m];
  s.b_up = at<float>(c.ws, c.p->off_bup) + net->poff[m];
  s.pstride = net->pstride;
  // per-neuron bias vector (layer 1: its bias plus the linear term of the bound)
  s.bias = at<float>(c.ws, c.p->off_bz) + net->poff[m];
  s.bias_hw = 1;
  (void)t;
  s.beta = at<float>(c.ws, c.p->off_beta);
  s.R = R;
  return s;
}

Sink bound_sink(const Chunk& c, long R, float* lo, float* hi, long bstride, long n_half) {
  Sink s{};
  // with a ReLU layer in front of T_1 the linear term was folded into the layer-1 bias (z1)
  s.x0 = c.net->L >= 2 ? nullptr : c.x0;
  s.eps = c.eps;
  s.beta = at<float>(c.ws, c.p->off_beta);
  s.R = R;
  s.lo = lo;
  s.hi = hi;
  s.bstride = bstride;
  s.n_half = n_half;
  return s;
}

int relax_layer(const Chunk& c, int m, const float* lsh = nullptr, const float* ush = nullptr) {
  const lirpa_net* net = c.net;
  long nm = net->n[m];
  long off = net->off[m];
  auto al = [](const void* ptr, uintptr_t a) { return ptr == nullptr || (uintptr_t)ptr % a == 0; };
  const bool vec4 = nm % 4 == 0 && net->n_relu % 4 == 0 && off % 4 == 0 &&
                    net->pstride % 4 == 0 && net->poff[m] % 4 == 0 && al(c.L, 16) &&
                    al(c.U, 16) && al(lsh, 16) && al(ush, 16) && al(c.alpha, 16) &&
                    al(c.split, 4) && al(c.ws, 256) && al(c.lp, 16) && al(c.up, 16);
  return launch_k(tag("relax_params", m, m), c.st, [&] {
    if (vec4) {
      hipLaunchKernelGGL(k_relax_params4, grid_for(c.nb * (nm / 4)), dim3(kBlock), 0, c.st,
                         c.nb, nm / 4, net->n_relu, off, net->pstride, net->poff[m], c.L, c.U,
                         lsh, ush, c.split, c.alpha, at<float>(c.ws, c.p->off_alo),
                         at<float>(c.ws, c.p->off_aup), at<float>(c.ws, c.p->off_bup),
                         at<int8_t>(c.ws, c.p->off_code), c.lp, c.up);
      return;
    }
    hipLaunchKernelGGL(k_relax_params, grid_for(c.nb * nm), dim3(kBlock), 0, c.st, c.nb, nm,
                       net->n_relu, off, net->pstride, net->poff[m], c.L, c.U, lsh, ush,
                       c.split, c.alpha,
                       at<float>(c.ws, c.p->off_alo), at<float>(c.ws, c.p->off_aup),
                       at<float>(c.ws, c.p->off_bup), at<int8_t>(c.ws, c.p->off_code), c.lp,
                       c.up);
  });
}

// Stages m = mtop .. 1 on rows already in slab 0 (relaxed onto layer mtop when mtop < L, raw
// spec rows when mtop == L), ending with the concretisation into (lo, hi).
float* tape_of(const Chunk& c, int pass, int m) {
  return c.tape ? at<float>(c.ws, c.p->off_tape[pass][m]) : nullptr;
}
// the pass's sign tape over x (one byte per entry, in the place of its tape over layer 0)
int8_t* tsign_of(const Chunk& c, int pass) {
  return c.tape ? at<int8_t>(c.ws, c.p->off_tape[pass][0]) : nullptr;
}

// k_convT_fc_bound for layers 1 and 2 of the net when they are convolutions of a covered
// geometry (fc: rows built from W_3; otherwise read from a slab, with nbs sub-domains per block
// at most); null otherwise.
using FcBoundKernel = void (*)(DLayer, DLayer, const float*, unsigned, unsigned, Sink, FcSrc);
// (spec: the variant that takes the final pass's spec rows from C W_L through a closing
// Linear layer of 97..100 features; conv 3 -> 8 -> 16 channels, three sub-domains per block;
// tape: the FC variant that also writes the reverse sweep's tape over g^(1) and sign tape)
FcBoundKernel conv12_bound_for(const lirpa_net* net, bool fc, int nbs, int* nwaves,
                               bool spec = false, bool tape = false) {
  if (net->L < 3) return nullptr;
  const lirpa_layer &t2 = net->T[1], &t1 = net->T[0];
  if (t2.kind != LIRPA_CONV2D || t1.kind != LIRPA_CONV2D) return nullptr;
  const bool t1_ok = t1.k == 4 && t1.stride == 2 && t1.pad == 1 && t1.in_c == 3 &&
                     t1.in_h == 32 && t1.in_w == 32 && t1.out_h == 16 && t1.out_w == 16;
  const bool t2_ok = t2.k == 4 && t2.stride == 2 && t2.pad == 1 && t2.in_h == 16 &&
                     t2.in_w == 16 && t2.out_h == 8 && t2.out_w == 8;
  if (!t1_ok || !t2_ok) return nullptr;
  if (t1.out_c == 8 && t2.in_c == 8 && t2.out_c == 16) {
    *nwaves = 8 / 2 + 4;
    if (spec) {
      // one g^(1) channel per matrix wave: 8 matrix waves, so that each takes one entry tile
      // of the spec source, its operands loaded a whole step ahead
      *nwaves = 8 + 4;
      return fc || nbs != 3
                 ? nullptr
                 : k_convT_fc_bound<4, 2, 1, 8, 8, 16, 16, 16, 8, 1, 4, 2, 1, 32, 32, 3, 4, false, 3,
                                    25>;
    }
    if (fc && tape)
      return k_convT_fc_bound<4, 2, 1, 8, 8, 16, 16, 16, 8, 2, 4, 2, 1, 32, 32, 3, 4, true, 2, 0,
                              true>;
    if (fc) return k_convT_fc_bound<4, 2, 1, 8, 8, 16, 16, 16, 8, 2, 4, 2, 1, 32, 32, 3, 4, true, 2>;
    if (nbs == 2)
      return k_convT_fc_bound<4, 2, 1, 8, 8, 16, 16, 16, 8, 2, 4, 2, 1, 32, 32, 3, 4, false, 2>;
    return k_convT_fc_bound<4, 2, 1, 8, 8, 16, 16, 16, 8, 2, 4, 2, 1, 32, 32, 3, 4, false, 3>;
  }
  // 3 -> 16 -> 32 channels: 8 matrix waves and 4 x waves, one block per CU (the slab source with three
  // sub-domains per block would not fit in LDS)
  if (t1.out_c == 16 && t2.in_c == 16 && t2.out_c == 32 && (fc || nbs == 2) && !spec) {
    *nwaves = 16 / 2 + 4;
    if (fc && tape)
      return k_convT_fc_bound<4, 2, 1, 8, 8, 16, 16, 32, 16, 2, 4, 2, 1, 32, 32, 3, 4, true, 2, 0,
                              true>;
    if (fc) return k_convT_fc_bound<4, 2, 1, 8, 8, 16, 16, 32, 16, 2, 4, 2, 1, 32, 32, 3, 4, true, 2>;
    return k_convT_fc_bound<4, 2, 1, 8, 8, 16, 16, 32, 16, 2, 4, 2, 1, 32, 32, 3, 4, false, 2>;
  }
  return nullptr;
}

// Fused last two stages (T_2^T + relaxation of layer 1, T_1^T + concretisation) when both
// layers are convolutions of a covered geometry; null otherwise.  *nwaves, *lds as launched.
using ConvT2Kernel = void (*)(DLayer, DLayer, const float*, unsigned, unsigned, Sink);
ConvT2Kernel convT2_bound_for(const lirpa_net* net, int* nwaves, size_t* lds) {
  if (net->L < 3) return nullptr;
  const lirpa_layer &a = net->T[0], &t = net->T[1];
  if (a.kind != LIRPA_CONV2D || t.kind != LIRPA_CONV2D) return nullptr;
  const bool t1_ok = a.k == 4 && a.stride == 2 && a.pad == 1 && a.in_c == 3 && a.in_h == 32 &&
                     a.in_w == 32 && a.out_h == 16 && a.out_w == 16 && a.out_c == 8;
  if (!t1_ok) return nullptr;
  auto set = [&](int co, int ci, int w1, int k, int s_, int ns) {
    const int rsl = s_ > k - s_ ? s_ : k - s_;
    const int cs = w1 * 16 + (80 - (w1 * 16) % 64) % 64;
    const int cs1 = 16 * 16 + 16;
    *nwaves = ci + ns + 3;
    *lds = (size_t)(2 * co * cs + 3 * rsl * ci * cs1 + 2 * 2 * 4 * rsl * ci * 16 + (ns + 3) * 16) *
           sizeof(float);
  };
  // T_2: Conv(8 -> 8, k3, s1, p1), 16x16 -> 16x16.  A stride-2 T_2 (8 -> 16 channels)
  // stays on the separate stage kernels: there each x wave carries twice the matrix work of a
  // T_2 wave per step, and at one block per CU that measured slower than the unfused pair.
  if (t.k == 3 && t.stride == 1 && t.pad == 1 && t.in_c == 8 && t.out_c == 8 && t.in_h == 16 &&
      t.out_h == 16 && t.out_w == 16) {
    set(8, 8, 16, 3, 1, 4);
    return k_convT2_bound<3, 1, 1, 16, 16, 16, 16, 8, 8, 4, 4, 2, 1, 32, 32, 3>;
  }
  return nullptr;
}

int run_stages(const Chunk& c, int pass, int mtop, long R, long Q, long ldq, float* lo,
               float* hi, long bstride, long n_half) {
  float* slab[2] = {at<float>(c.ws, c.p->off_slab0), at<float>(c.ws, c.p->off_slab1)};
  int cur = 0;
  for (int m = mtop; m >= 1; --m) {
    int e;
    if (m == 2 && !c.tape && R >= 8) {
      // T_2^T, the layer-1 relaxation, T_1^T and the concretisation in one kernel
      int nw = 0;
      if (FcBoundKernel kern = conv12_bound_for(c.net, false, R >= 16 ? 2 : 3, &nw)) {
        Sink s = slab_sink(c, 1, nullptr, ldq, R);
        const Sink sb = bound_sink(c, R, lo, hi, bstride, n_half);
        s.eps = sb.eps;
        s.x0 = sb.x0;
        s.lo = sb.lo;
        s.hi = sb.hi;
        s.bstride = sb.bstride;
        s.n_half = sb.n_half;
        const unsigned nblk16 = (unsigned)round_up((Q + 15) / 16, 16);
        return launch_k(tag("convT_slab_bound", 2, pass), c.st, [&] {
          hipLaunchKernelGGL(kern, dim3(nblk16), dim3(64 * nw), 0, c.st,
                             dlayer(c.net->T[1]), dlayer(c.net->T[0]), slab[cur],
                             (unsigned)ldq, (unsigned)Q, s, FcSrc{});
        });
      }
    }
    if (m == 2 && !c.tape && R >= 16) {
      int nw = 0;
      size_t lds = 0;
      if (ConvT2Kernel kern = convT2_bound_for(c.net, &nw, &lds)) {
        Sink s = slab_sink(c, 1, nullptr, ldq, R);
        Sink sb = bound_sink(c, R, lo, hi, bstride, n_half);
        s.eps = sb.eps;
        s.x0 = sb.x0;
        s.lo = sb.lo;
        s.hi = sb.hi;
        s.bstride = sb.bstride;
        s.n_half = sb.n_half;
        s.ldq = ldq;
        const unsigned nblk16 = (unsigned)round_up((Q + 15) / 16, 16);
        if (lds > 65536 &&
            hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds) != hipSuccess)
          return fail(LIRPA_EDEVICE, "cannot reserve %zu bytes of LDS", lds);
        return launch_k(tag("convT2_bound", 2, pass), c.st, [&] {
          hipLaunchKernelGGL(kern, dim3(nblk16), dim3(64 * nw), lds, c.st,
                             dlayer(c.net->T[1]), dlayer(c.net->T[0]), slab[cur], (unsigned)ldq,
                             (unsigned)Q, s);
        });
      }
    }
    if (m > 1) {
      Sink s = slab_sink(c, m - 1, slab[1 - cur], ldq, R);
      s.tape = tape_of(c, pass, m - 1);
      e = launch_stage<MODE_SLAB>(c.net, m, pass, slab[cur], ldq, Q, s, c.st);
      cur ^= 1;
    } else {
      Sink s = bound_sink(c, R, lo, hi, bstride, n_half);
      s.ldq = ldq;
      s.tsign = tsign_of(c, pass);
      e = launch_stage<MODE_BOUND>(c.net, m, pass, slab[cur], ldq, Q, s, c.st);
    }
    if (e) return e;
  }
  return LIRPA_OK;
}

// Returns 1 when the shapes do not qualify (the caller runs the dense pass).
int pass2_window(const Chunk& c) {
  const lirpa_net* net = c.net;
  int nw = 0;
  Pass2Kernel kern = pass2_kernel_for(net, &nw);
  if (!kern) return 1;
  const lirpa_layer &t1 = net->T[0], &t2 = net->T[1];
  long blocks = pass2_blocks(net, c.nb) / p2_xw(net);
  const float* alo = at<float>(c.ws, c.p->off_alo) + net->poff[1];
  const float* aup = at<float>(c.ws, c.p->off_aup) + net->poff[1];
  const float* bup = at<float>(c.ws, c.p->off_bup) + net->poff[1];
  const size_t p2 = (size_t)net->poff[2];
  return launch_k(tag("pass2_window", 1, 2), c.st, [&] {
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64 * nw), 0, c.st, dlayer(t1),
                       dlayer(t2), c.nb, alo, aup, bup, net->pstride,
                       at<float>(c.ws, c.p->off_z1), c.eps, c.L, c.U, net->n_relu, net->off[2],
                       c.split, c.alpha, at<float>(c.ws, c.p->off_alo) + p2,
                       at<float>(c.ws, c.p->off_aup) + p2, at<float>(c.ws, c.p->off_bup) + p2,
                       at<int8_t>(c.ws, c.p->off_code), c.lp, c.up);
  });
}

// Kernel for the receptive-field pass 3 (T_3, T_2 stride-1 convolutions over T_1), or null.
using Pass3Kernel = void (*)(DLayer, DLayer, DLayer, const float*, const float*, const float*,
                             long, long, long, const float*, float, float*, float*, long, long);
Pass3Kernel pass3_kernel_for(const lirpa_net* net) {
  if (net->L < 4) return nullptr;
  const lirpa_layer &t1 = net->T[0], &t2 = net->T[1], &t3 = net->T[2];
  if (t1.kind != LIRPA_CONV2D || t2.kind != LIRPA_CONV2D || t3.kind != LIRPA_CONV2D)
    return nullptr;
  if (t3.out_c % 16 && t3.out_c != 8) return nullptr;
  const bool s1 = t1.k == 4 && t1.stride == 2 && t1.pad == 1 && t1.out_c == 8;
  const bool s2 = t2.k == 3 && t2.stride == 1 && t2.pad == 1 && t2.out_c == 8;
  const bool s3 = t3.k == 3 && t3.stride == 1 && t3.pad == 1;
  if (s1 && s2 && s3 && t1.in_c <= 8) return k_pass3_window<3, 1, 3, 1, 4, 2, 1, 8, 8>;
  return nullptr;
}

int pass3_window(const Chunk& c) {
  const lirpa_net* net = c.net;
  Pass3Kernel kern = pass3_kernel_for(net);
  if (!kern) return 1;
  const lirpa_layer& t3 = net->T[2];
  long blocks = c.nb * p2_groups(t3.out_c) * t3.out_h * t3.out_w;
  return launch_k(tag("pass3_window", 1, 3), c.st, [&] {
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(512), 0, c.st, dlayer(net->T[0]),
                       dlayer(net->T[1]), dlayer(net->T[2]), at<float>(c.ws, c.p->off_alo),
                       at<float>(c.ws, c.p->off_aup), at<float>(c.ws, c.p->off_bup),
                       net->pstride, net->poff[1], net->poff[2], at<float>(c.ws, c.p->off_bz),
                       c.eps, c.L, c.U, net->n_relu, net->off[3]);
  });
}

// Witness forward kernels of the covered convolution shapes (the k4 s2 p1 and k3 s1 p1 layers
// of the convolution kernels); null for any other layer (the generic k_fwd_mfma runs).
using FwdKernel = void (*)(DLayer, const float*, unsigned, unsigned, long, const float*,
                           const float*, float, const float*, const float*, const float*,
                           const float*, long, float*, float*, float*, unsigned char*,
                           const float*, int, int);
template <int K, int S, int P, int CI, int CO, int HI, int WI, int HO, int WO>
FwdKernel fwd_conv_inst(bool witness, bool zout) {
  if (zout)
    return witness ? k_fwd_conv<K, S, P, CI, CO, HI, WI, HO, WO, true, true>
                   : k_fwd_conv<K, S, P, CI, CO, HI, WI, HO, WO, false, true>;
  return witness ? k_fwd_conv<K, S, P, CI, CO, HI, WI, HO, WO, true, false>
                 : k_fwd_conv<K, S, P, CI, CO, HI, WI, HO, WO, false, false>;
}
FwdKernel fwd_conv_for(const lirpa_layer& t, bool witness, bool zout) {
  if (t.kind != LIRPA_CONV2D) return nullptr;
  auto is = [&](int k, int s_, int p_, int ci, int co, int hi, int ho) {
    return t.k == k && t.stride == s_ && t.pad == p_ && t.in_c == ci && t.out_c == co &&
           t.in_h == hi && t.in_w == hi && t.out_h == ho && t.out_w == ho;
  };
  if (is(4, 2, 1, 3, 8, 32, 16)) return fwd_conv_inst<4, 2, 1, 3, 8, 32, 32, 16, 16>(witness, zout);
  if (is(4, 2, 1, 3, 16, 32, 16)) return fwd_conv_inst<4, 2, 1, 3, 16, 32, 32, 16, 16>(witness, zout);
  if (is(4, 2, 1, 8, 16, 16, 8)) return fwd_conv_inst<4, 2, 1, 8, 16, 16, 16, 8, 8>(witness, zout);
  if (is(4, 2, 1, 16, 32, 16, 8)) return fwd_conv_inst<4, 2, 1, 16, 32, 16, 16, 8, 8>(witness, zout);
  if (is(4, 2, 1, 8, 8, 16, 8)) return fwd_conv_inst<4, 2, 1, 8, 8, 16, 16, 8, 8>(witness, zout);
  if (is(3, 1, 1, 8, 8, 16, 16)) return fwd_conv_inst<3, 1, 1, 8, 8, 16, 16, 16, 16>(witness, zout);
  return nullptr;
}

// First stage of a bound pass k that opens at a fully connected layer k over a convolution
// k-1: the stage through T_{k-1} builds its input rows from W_k and the relaxation of layer k-1
// itself and writes the rows relaxed onto layer k-2 into slab 0.  Returns 1 when the shapes or
// alignment do not qualify (the caller runs the pass initialisation and the plain stage).
// Whether pass k (R rows per sub-domain) opens inside the stage through layer k-1.  With a
// gradient tape the pass then records no tape over g^(k-1): its rows are +-W_k[j] of every
// sub-domain, and the witness forward through layer k-1 reads them from W_k (which needs the
// fused forward kernel for that layer).
bool fc_open_ok(const Chunk& c, int k, long R) {
  const lirpa_net* net = c.net;
  if (k < 3 || k >= net->L || R < 16 || R % 2) return false;
  const lirpa_layer &fl = net->T[k - 1], &cv = net->T[k - 2];
  if (fl.kind != LIRPA_LINEAR || cv.kind != LIRPA_CONV2D) return false;
  if (reinterpret_cast<uintptr_t>(fl.W) % 16) return false;
  // parameter offsets of the kernel are 32-bit
  if ((double)c.nb * net->pstride >= 4.0e9) return false;
  int nw = 0;
  size_t lds = 0;
  if (!convT_ws_for(dlayer(cv), c.tape, true, &nw, &lds)) return false;
  if (c.tape && (R % 8 || !c.p->off_gpart || !fwd_conv_for(cv, k - 1 == 1, false))) return false;
  return true;
}

int fc_open_stage(const Chunk& c, int k, long R, long Q, long ldq) {
  const lirpa_net* net = c.net;
  if (!fc_open_ok(c, k, R)) return 1;
  const lirpa_layer &fl = net->T[k - 1], &cv = net->T[k - 2];
  int nw = 0;
  size_t lds = 0;
  DLayer t = dlayer(cv);
  WsKernel kern = convT_ws_for(t, c.tape, true, &nw, &lds);
  Sink s = slab_sink(c, k - 2, at<float>(c.ws, c.p->off_slab0), ldq, R);
  s.tape = tape_of(c, k, k - 2);
  FcSrc f{};
  f.W = fl.W;
  f.b = fl.b;
  f.nk = (int)net->n[k];
  f.a_lo = at<float>(c.ws, c.p->off_alo) + net->poff[k - 1];
  f.a_up = at<float>(c.ws, c.p->off_aup) + net->poff[k - 1];
  f.b_up = at<float>(c.ws, c.p->off_bup) + net->poff[k - 1];
  const unsigned nblk16 = (unsigned)round_up((Q + 15) / 16, 16);
  return launch_k(tag("convT_relax_fc", k - 1, k), c.st, [&] {
    hipLaunchKernelGGL(kern, dim3(nblk16), dim3(64 * nw), lds, c.st, t, nullptr, (unsigned)ldq,
                       (unsigned)Q, s, f);
  });
}

// Pass 3 of a net whose layers 1 and 2 are such convolutions and whose layer 3 is fully
// connected, bounded without a gradient tape: one kernel from the rows of W_3 to the bounds.
FcBoundKernel fc_bound_for(const lirpa_net* net, int k, int* nwaves, bool tape = false) {
  if (k != 3 || net->L < 4 || net->T[2].kind != LIRPA_LINEAR) return nullptr;
  return conv12_bound_for(net, true, 2, nwaves, false, tape);
}

// Whether pass k of a gradient chunk runs as one tape-writing k_convT_fc_bound.  Its rows are
// then interleaved (row 2j: +e_j, row 2j + 1: -e_j) and the reverse sweep of the pass runs
// k_fwd_conv12, which reads the two tapes that kernel writes.
bool fused_tape_pass(const Chunk& c, int k, long R) {
  int nw = 0;
  return c.tape && k == 3 && R % 8 == 0 && fc_open_ok(c, k, R) && c.p->off_gpart &&
         c.p->off_gpart2 && fwd12_for(c.net) && fc_bound_for(c.net, k, &nw, true);
}

// Returns 1 when the pass does not qualify (the caller runs the stages one by one).
int fc_bound_stage(const Chunk& c, int k, long R, long Q) {
  const lirpa_net* net = c.net;
  int nw = 0;
  const bool tape = c.tape;
  FcBoundKernel kern = fc_bound_for(net, k, &nw, tape);
  if (!kern || !fc_open_ok(c, k, R) || (tape && !fused_tape_pass(c, k, R))) return 1;
  const lirpa_layer& fl = net->T[k - 1];
  Sink s = slab_sink(c, 1, nullptr, 0, R);  // the relaxation of layer 1 (bias: z1)
  const Sink sb = bound_sink(c, R, c.L + net->off[k], c.U + net->off[k], net->n_relu, net->n[k]);
  s.eps = sb.eps;
  s.x0 = sb.x0;
  s.lo = sb.lo;
  s.hi = sb.hi;
  s.bstride = sb.bstride;
  s.n_half = sb.n_half;
  FcSrc f{};
  f.W = fl.W;
  f.b = fl.b;
  f.nk = (int)net->n[k];
  f.a_lo = at<float>(c.ws, c.p->off_alo) + net->poff[k - 1];
  f.a_up = at<float>(c.ws, c.p->off_aup) + net->poff[k - 1];
  f.b_up = at<float>(c.ws, c.p->off_bup) + net->poff[k - 1];
  f.split = c.split;
  f.alpha = c.alpha;
  f.r_lo = at<float>(c.ws, c.p->off_alo) + net->poff[k];
  f.r_up = at<float>(c.ws, c.p->off_aup) + net->poff[k];
  f.r_bu = at<float>(c.ws, c.p->off_bup) + net->poff[k];
  f.code = at<int8_t>(c.ws, c.p->off_code);
  f.n_relu = net->n_relu;
  f.off = net->off[k];
  f.lpar = c.lp;
  f.upar = c.up;
  const long ldq = round_up(Q, 64);
  if (tape) {
    s.tape = tape_of(c, k, 1);
    s.tsign = tsign_of(c, k);
  }
  const unsigned nblk16 = (unsigned)round_up((Q + 15) / 16, 16);
  return launch_k(tag("convT_fc_bound", k - 1, k), c.st, [&] {
    hipLaunchKernelGGL(kern, dim3(nblk16), dim3(64 * nw), 0, c.st, dlayer(net->T[k - 2]),
                       dlayer(net->T[0]), nullptr, tape ? (unsigned)ldq : 0u, (unsigned)Q, s, f);
  });
}

// Kernel for the receptive-field pass 4 (T_4 over the stride-1 T_3, T_2 over T_1, 8 channels
// each), or null.
using Pass4Kernel = void (*)(DLayer, DLayer, DLayer, DLayer, const float*, const float*,
                             const float*, long, long, long, long, const float*, float, float*,
                             float*, long, long);
Pass4Kernel pass4_kernel_for(const lirpa_net* net) {
  if (net->L < 5) return nullptr;
  const lirpa_layer &t1 = net->T[0], &t2 = net->T[1], &t3 = net->T[2], &t4 = net->T[3];
  for (const lirpa_layer* t : {&t1, &t2, &t3, &t4})
    if (t->kind != LIRPA_CONV2D) return nullptr;
  if (t4.out_c % 16 && t4.out_c != 8) return nullptr;
  const bool s1 = t1.k == 4 && t1.stride == 2 && t1.pad == 1 && t1.out_c == 8 && t1.in_c <= 8;
  const bool s2 = t2.k == 3 && t2.stride == 1 && t2.pad == 1 && t2.out_c == 8;
  const bool s3 = t3.k == 3 && t3.stride == 1 && t3.pad == 1 && t3.out_c == 8;
  const bool s4 = t4.k == 4 && t4.stride == 2 && t4.pad == 1;
  if (s1 && s2 && s3 && s4) return k_pass4_window<4, 2, 1, 3, 1, 3, 1, 4, 2, 1, 8, 8, 8>;
  return nullptr;
}

bool pass_on_chip(const lirpa_net* net, int k, long Bc) {
  // the same choices, in the same order, as bound_chunk makes for a chunk without a tape
  int nw = 0;
  if (k == 2) return pass2_kernel_for(net, &nw) != nullptr;
  if (k == 4 && pass4_kernel_for(net)) return true;
  if (k == 3 && pass3_kernel_for(net)) return true;
  if (!fc_bound_for(net, k, &nw)) return false;
  // fc_open_ok holds for every chunk of at most Bc sub-domains when it holds for Bc
  Chunk c{};
  c.net = net;
  c.nb = Bc;
  c.tape = false;
  return fc_open_ok(c, k, 2 * net->n[k]);
}

int pass4_window(const Chunk& c) {
  const lirpa_net* net = c.net;
  Pass4Kernel kern = pass4_kernel_for(net);
  if (!kern) return 1;
  const lirpa_layer& t4 = net->T[3];
  long blocks = c.nb * p2_groups(t4.out_c) * t4.out_h * t4.out_w;
  return launch_k(tag("pass4_window", 1, 4), c.st, [&] {
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(512), 0, c.st, dlayer(net->T[0]),
                       dlayer(net->T[1]), dlayer(net->T[2]), dlayer(net->T[3]),
                       at<float>(c.ws, c.p->off_alo), at<float>(c.ws, c.p->off_aup),
                       at<float>(c.ws, c.p->off_bup), net->pstride, net->poff[1], net->poff[2],
                       net->poff[3], at<float>(c.ws, c.p->off_bz), c.eps, c.L, c.U, net->n_relu,
                       net->off[4]);
  });
}

int bound_chunk(const Chunk& c, const float* C, float* lb) {
  const lirpa_net* net = c.net;
  const int L = net->L;
  long n1 = net->n[1];
  if (L >= 2) {
    // layer 1: the shared exact bounds, copied into every sub-domain's rows on the way
    const float* l1u1 = at<float>(c.ws, c.p->off_l1u1);
    if (int e = relax_layer(c, 1, l1u1, l1u1 + n1)) return e;
  }
  for (int k = 2; k <= L - 1; ++k) {
    long nk = net->n[k], R = 2 * nk, Q = c.nb * R, ldq = round_up(Q, 64);
    if (k == 2 && (!c.tape || pass2_grad_kernel_for(net))) {
      int e = pass2_window(c);
      if (e != 1) {
        if (e) return e;  // (the kernel also wrote the relaxation of layer 2)
        continue;
      }
    }
    if (k == 4 && !c.tape) {
      int e = pass4_window(c);
      if (e != 1) {
        if (e) return e;
        if (int e2 = relax_layer(c, k)) return e2;
        continue;
      }
    }
    if (k == 3 && !c.tape) {
      int e = pass3_window(c);
      if (e != 1) {
        if (e) return e;
        if (int e2 = relax_layer(c, k)) return e2;
        continue;
      }
    }
    {
      int e = fc_bound_stage(c, k, R, Q);
      if (e != 1) {
        if (e) return e;  // (the kernel also wrote the relaxation of layer k)
        continue;
      }
    }
    {
      int e = fc_open_stage(c, k, R, Q, ldq);
      if (e != 1) {
        if (e) return e;
        if (int e2 = run_stages(c, k, k - 2, R, Q, ldq, c.L + net->off[k], c.U + net->off[k],
                                net->n_relu, nk))
          return e2;
        if (int e2 = relax_layer(c, k)) return e2;
        continue;
      }
    }
    Sink s = slab_sink(c, k - 1, at<float>(c.ws, c.p->off_slab0), ldq, R);
    s.tape = tape_of(c, k, k - 1);
    const float* wT = c.p->off_wT[k] ? at<float>(c.ws, c.p->off_wT[k]) : nullptr;
    if (int e = launch_k(tag("init_rows", k, k), c.st, [&] {
          if (wT)
            hipLaunchKernelGGL(k_init_fc_rows, dim3((unsigned)((Q + 63) / 64)), dim3(256), 0,
                               c.st, dlayer(net->T[k - 1]), wT, Q, s);
          else
            hipLaunchKernelGGL(k_init_rows<MODE_SLAB>, grid_for(Q), dim3(kBlock), 0, c.st,
                               dlayer(net->T[k - 1]), wT, Q, s);
        }))
      return e;
    if (int e = run_stages(c, k, k - 1, R, Q, ldq, c.L + net->off[k], c.U + net->off[k],
                           net->n_relu, nk))
      return e;
    if (int e = relax_layer(c, k)) return e;
  }
  // final pass
  long R = c.S, Q = c.nb * R, ldq = round_up(Q, 64);
  const lirpa_layer& tL = net->T[L - 1];
  if (!c.tape && L == 4 && c.p->off_wsp && net->T[2].kind == LIRPA_LINEAR && R >= 8 &&
      (net->n[3] + 3) / 4 == 25) {
    // the whole final pass in one kernel: the spec rows through T_4 (k_setup's C W_4), their
    // relaxation onto layer 3, T_3^T on MFMA and the relaxation onto layer 2 built into the
    // conv kernel's input tile, then T_2^T, the layer-1 relaxation, T_1^T and the
    // concretisation (conv 3 -> 8 -> 16 channels on 32x32, then a Linear layer of 97..100)
    int nw = 0;
    if (FcBoundKernel kern = conv12_bound_for(net, false, 3, &nw, /*spec=*/true)) {
      Sink s = slab_sink(c, 1, nullptr, ldq, R);
      const Sink sb = bound_sink(c, R, lb, lb, c.S, c.S);
      s.eps = sb.eps;
      s.x0 = sb.x0;
      s.lo = sb.lo;
      s.hi = sb.hi;
      s.bstride = sb.bstride;
      s.n_half = sb.n_half;
      FcSrc f{};
      f.W = net->T[2].W;
      f.b = at<float>(c.ws, c.p->off_wsp);
      f.nk = (int)net->n[3];
      f.a_lo = at<float>(c.ws, c.p->off_alo) + net->poff[2];
      f.a_up = at<float>(c.ws, c.p->off_aup) + net->poff[2];
      f.b_up = at<float>(c.ws, c.p->off_bup) + net->poff[2];
      f.r_lo = at<float>(c.ws, c.p->off_alo) + net->poff[3];
      f.r_up = at<float>(c.ws, c.p->off_aup) + net->poff[3];
      f.r_bu = at<float>(c.ws, c.p->off_bup) + net->poff[3];
      f.sbias_k = at<float>(c.ws, c.p->off_bz) + net->poff[2];
      f.sbias_k1 = at<float>(c.ws, c.p->off_bz) + net->poff[3];
      const unsigned nblk16 = (unsigned)round_up((Q + 15) / 16, 16);
      return launch_k(tag("spec_bound", 2, L), c.st, [&] {
        hipLaunchKernelGGL(kern, dim3(nblk16), dim3(64 * nw), 0, c.st, dlayer(net->T[1]),
                           dlayer(net->T[0]), nullptr, (unsigned)ldq, (unsigned)Q, s, f);
      });
    }
  }
  if (!c.tape && L >= 3 && c.p->off_wsp && net->T[L - 2].kind == LIRPA_LINEAR) {
    // the spec rows through T_L and T_{L-1} in one kernel
    constexpr int NW = 16;
    Sink s = slab_sink(c, L - 2, at<float>(c.ws, c.p->off_slab0), ldq, R);
    const long nj = net->n[L - 1];
    const size_t lds = (size_t)(((nj + 3) & ~3L) * 16 + NW * 64 + NW * 16) * sizeof(float);
    // k-steps of the kernel: ceil(n_{L-1} / 4) for the instantiated sizes
    auto fkern = [&]() -> void (*)(DLayer, const float*, int, long, long, const float*,
                                   const float*, const float*, const float*, Sink) {
      switch ((nj + 3) / 4) {
        case 8: return k_final_fc<NW, 8>;
        case 16: return k_final_fc<NW, 16>;
        case 25: return k_final_fc<NW, 25>;
        case 32: return k_final_fc<NW, 32>;
        default: return nullptr;
      }
    };
    if (lds <= 65536 && fkern()) {
      const size_t po = (size_t)net->poff[L - 1];
      if (int e = launch_k(tag("final_fc", L - 1, L), c.st, [&] {
            hipLaunchKernelGGL(fkern(), dim3((unsigned)((Q + 15) / 16)), dim3(64 * NW),
                               lds, c.st, dlayer(net->T[L - 2]),
                               at<float>(c.ws, c.p->off_wsp), (int)c.S, c.nb,
                               Q, at<float>(c.ws, c.p->off_alo) + po,
                               at<float>(c.ws, c.p->off_aup) + po,
                               at<float>(c.ws, c.p->off_bup) + po,
                               at<float>(c.ws, c.p->off_bz) + po, s);
          }))
        return e;
      return run_stages(c, L, L - 2, R, Q, ldq, lb, lb, c.S, c.S);
    }
  }
  if (int e = launch_k(tag("spec_rows", L, L), c.st, [&] {
        hipLaunchKernelGGL(k_spec_rows, grid_for(Q), dim3(kBlock), 0, c.st, C, net->n[L], tL.b,
                           tL.out_h * tL.out_w, Q, c.S, at<float>(c.ws, c.p->off_slab0), ldq,
                           at<float>(c.ws, c.p->off_beta));
      }))
    return e;
  return run_stages(c, L, L, R, Q, ldq, lb, lb, c.S, c.S);
}

// Exact layer-1 bounds, shared by every sub-domain: rows +-e_j of h^(1) through T_1, then
// concretised (no relaxation in front of layer 1).
int layer1_bounds(const lirpa_net* net, const Plan& p, void* ws, const float* x0, float eps,
                  const float* C, int S, hipStream_t st) {
  long n1 = net->n[1];
  SetupJob job{};
  job.t1 = dlayer(net->T[0]);
  job.x0 = x0;
  job.eps = eps;
  job.l1 = at<float>(ws, p.off_l1u1);
  job.z1 = at<float>(ws, p.off_z1);
  job.n1 = n1;
  long total = 16 * n1;
  for (int m = 2; m <= net->L - 1; ++m) {  // bias vectors (layer 1's is z1)
    const lirpa_layer& t = net->T[m - 1];
    job.fill_n[job.nfill] = net->n[m];
    job.fill_hw[job.nfill] = t.out_h * t.out_w;
    job.fill_b[job.nfill] = t.b;
    job.fill_out[job.nfill] = at<float>(ws, p.off_bz) + net->poff[m];
    total += net->n[m];
    ++job.nfill;
  }
  // transposed FC weights, for the passes that do not open inside the stage below (those read
  // W_k row by row); that holds for every chunk if it holds for the largest
  Chunk cp{};
  cp.net = net;
  cp.p = &p;
  cp.nb = p.Bc;
  cp.tape = p.mode == 1;
  for (int k = 2; k <= net->L - 1; ++k) {
    if (!p.off_wT[k] || fc_open_ok(cp, k, 2 * net->n[k])) continue;
    const lirpa_layer& t = net->T[k - 1];
    job.tr_W[job.ntr] = t.W;
    job.tr_out[job.ntr] = t.out_c;
    job.tr_in[job.ntr] = t.in_c;
    job.tr_dst[job.ntr] = at<float>(ws, p.off_wT[k]);
    total += (long)t.out_c * t.in_c;
    ++job.ntr;
  }
  if (p.off_wsp) {
    job.wsp = at<float>(ws, p.off_wsp);
    job.C = C;
    job.tL = dlayer(net->T[net->L - 1]);
    job.S = S;
    total += (long)S * (net->n[net->L - 1] + 1);
  }
  return launch_k(tag("setup", 1, 1), st, [&] {
    hipLaunchKernelGGL(k_setup, grid_for(total), dim3(kBlock), 0, st, job);
  });
}

// Gradient of J_b = sum_s lb[b][s] with respect to alpha for every sub-domain of the chunk,
// after bound_chunk has recorded the tape (passes visited in descending order; the adjoints of
// l^(P), u^(P) are complete once every later pass has been visited).  full == 0 visits the
// final pass only (intermediate bounds held fixed).  Result in ga ([nb][n_relu]).
int grad_chunk(const Chunk& c, int full) {
  const lirpa_net* net = c.net;
  const Plan& p = *c.p;
  const int L = net->L;
  long per = c.nb * net->n_relu;
  float* ga = at<float>(c.ws, p.off_ga);
  float* gl = at<float>(c.ws, p.off_gl);
  float* gu = at<float>(c.ws, p.off_gu);
  float* w = at<float>(c.ws, p.off_w);
  float* za = at<float>(c.ws, p.off_za);
  float* zb = at<float>(c.ws, p.off_zb);
  float* G = at<float>(c.ws, p.off_G);
  // (workspace regions: 256-byte aligned)
  if (int e = launch_k("zero", c.st, [&] {
        hipLaunchKernelGGL(k_zero3, grid_for((per + 3) / 4), dim3(kBlock), 0, c.st, per, ga, gl,
                           gu);
      }))
    return e;
  bool have_list1 = false;  // k_unstable_index has listed the layer-1 neurons of this chunk
  for (int P = L; P >= 2; --P) {
    if (!full && P < L) break;
    if (P == 2 && P < L) {
      if (Pass2GradKernel gk = pass2_grad_kernel_for(net)) {
        const lirpa_layer &t1 = net->T[0], &t2 = net->T[1];
        long blocks = pass2_blocks(net, c.nb) / p2_xw(net);  // windows / windows per block
        float* part = at<float>(c.ws, p.off_p2part);
        unsigned char* pflag = at<unsigned char>(c.ws, p.off_p2flag);
        const int8_t* code = at<int8_t>(c.ws, p.off_code);
        int e = launch_k(tag("pass2_window_grad", 1, 2), c.st, [&] {
          hipLaunchKernelGGL(gk, dim3((unsigned)blocks), dim3(64 * t1.in_c), 0, c.st, dlayer(t1),
                             dlayer(t2), at<float>(c.ws, p.off_alo) + net->poff[1],
                             at<float>(c.ws, p.off_aup) + net->poff[1], net->pstride, c.eps, gl,
                             gu, code, net->n_relu, net->off[2], at<float>(c.ws, p.off_z1), part,
                             pflag);
        });
        if (e) return e;
        long n1 = net->n[1];
        e = launch_k(tag("pass2_grad_gather", 1, 2), c.st, [&] {
          if (have_list1)  // the sub-domains' unstable layer-1 neurons are listed (pass 3)
            hipLaunchKernelGGL(k_pass2_grad_gather_c, dim3((unsigned)c.nb), dim3(kBlock), 0,
                               c.st, dlayer(t1), dlayer(t2), t2.k * t2.k, part, pflag,
                               at<int>(c.ws, p.off_list1), at<int>(c.ws, p.off_cnt1), n1,
                               net->n_relu, ga);
          else
            hipLaunchKernelGGL(k_pass2_grad_gather, grid_for(c.nb * n1), dim3(kBlock), 0, c.st,
                               c.nb, dlayer(t1), dlayer(t2), t2.k * t2.k, part, pflag, code,
                               net->n_relu, ga);
        });
        if (e) return e;
        continue;
      }
    }
    long R = (P < L) ? 2 * net->n[P] : c.S, Q = c.nb * R, ldq = round_up(Q, 64);
    long offP = (P < L) ? net->off[P] : 0;
    // rows of a pass bounded by the tape-writing k_convT_fc_bound are interleaved
    const bool inter = P < L && fused_tape_pass(c, P, R);
    if (int e = launch_k(tag("row_weights", P, P), c.st, [&] {
          hipLaunchKernelGGL(k_row_weights, grid_for(Q), dim3(kBlock), 0, c.st, Q, R, net->n[P],
                             net->n_relu, offP, (int)(P == L), (int)inter, gl, gu, w);
        }))
      return e;
    if (P == 3 && P < L && R % 8 == 0 && p.off_gpart && p.off_gpart2 && fc_open_ok(c, P, R)) {
      if (Fwd12Kernel fk = fwd12_for(net)) {
        // both convolutions of pass 3's witness forward in one kernel, then both layers' sums
        const lirpa_layer &t1 = net->T[0], &t2 = net->T[1];
        float* part1 = at<float>(c.ws, p.off_gpart);
        float* part2 = at<float>(c.ws, p.off_gpart2);
        unsigned char* gflag = at<unsigned char>(c.ws, p.off_gflag);
        // T_2's weights with the tap indices exchanged (the kernel's per-tile operand loads)
        float* w2t = at<float>(c.ws, p.off_w2t);
        const long nw2 = (long)t2.out_c * t2.in_c * t2.k * t2.k;
        if (int e = launch_k(tag("taps_swap", 2, P), c.st, [&] {
              hipLaunchKernelGGL(k_taps_swap, grid_for(nw2), dim3(kBlock), 0, c.st, nw2, t2.k,
                                 t2.W, w2t);
            }))
          return e;
        // with 32 channels the kernel reads T_3's weights channel-last, and writes its layer-1
        // sums for the unstable neurons only, at their ranks
        const float* w3 = net->T[2].W;
        int* kidx1 = at<int>(c.ws, p.off_kidx1);
        int* list1 = at<int>(c.ws, p.off_list1);
        int* cnt1 = at<int>(c.ws, p.off_cnt1);
        int* kidx2 = at<int>(c.ws, p.off_kidx2);
        int* list2 = at<int>(c.ws, p.off_list2);
        int* cnt2 = at<int>(c.ws, p.off_cnt2);
        unsigned* psel = at<unsigned>(c.ws, p.off_psel);
        if (t2.out_c == 32) {
          have_list1 = true;  // (pass 2's gather below takes the layer-1 list too)
          for (int m = 1; m <= 2; ++m)
            if (int e = launch_k(tag("unstable_index", m, P), c.st, [&] {
                  hipLaunchKernelGGL(k_unstable_index, dim3((unsigned)c.nb), dim3(256), 0, c.st,
                                     (int)net->n[m], at<int8_t>(c.ws, p.off_code) + net->off[m],
                                     net->n_relu, m == 1 ? kidx1 : kidx2, m == 1 ? list1 : list2,
                                     m == 1 ? cnt1 : cnt2);
                }))
              return e;
          if (int e = launch_k(tag("pair_select", 2, P), c.st, [&] {
                hipLaunchKernelGGL(k_pair_select, dim3((unsigned)c.nb), dim3(256), 0, c.st,
                                   at<int8_t>(c.ws, p.off_code) + net->off[2],
                                   (unsigned)net->n_relu, psel);
              }))
            return e;
          float* w3c = at<float>(c.ws, p.off_w3c);
          const lirpa_layer& t3 = net->T[2];
          const long nw3 = (long)t3.out_c * t3.in_c;
          if (int e = launch_k(tag("fc_chlast", 3, P), c.st, [&] {
                hipLaunchKernelGGL(k_fc_chlast, grid_for(nw3), dim3(kBlock), 0, c.st, nw3,
                                   t2.out_c, t2.out_h * t2.out_w, t3.W, w3c);
              }))
            return e;
          w3 = w3c;
        }
        const unsigned nblk8 = (unsigned)round_up((Q + 7) / 8, 8);
        if (int e = launch_k(tag("fwd12", 1, P), c.st, [&] {
              hipLaunchKernelGGL(fk, dim3(nblk8), dim3(256), 0, c.st, dlayer(t1), dlayer(t2),
                                 tsign_of(c, P), (unsigned)ldq, (unsigned)Q, (unsigned)R, w,
                                 c.x0, c.eps, tape_of(c, P, 1),
                                 at<float>(c.ws, p.off_alo) + net->poff[1],
                                 at<float>(c.ws, p.off_aup) + net->poff[1],
                                 at<float>(c.ws, p.off_bup) + net->poff[1],
                                 (unsigned)net->pstride, w3, (unsigned)net->n[3],
                                 (unsigned)inter, psel, kidx1, kidx2, w2t, part1, part2, gflag);
            }))
          return e;
        for (int m = 1; m <= 2; ++m) {
          const lirpa_layer& t = net->T[m - 1];
          const long off = net->off[m];
          if (int e = launch_k(tag("grad_gather", m, P), c.st, [&] {
                if (t2.out_c == 32)
                  hipLaunchKernelGGL(k_grad_gather_c, dim3((unsigned)c.nb), dim3(kBlock), 0,
                                     c.st, net->n[m], R, m == 1 ? part1 : part2, gflag,
                                     m == 1 ? list1 : list2, m == 1 ? cnt1 : cnt2, c.L + off,
                                     c.U + off, net->n_relu, ga + off, gl + off, gu + off);
                else
                  hipLaunchKernelGGL(k_grad_gather, grid_for(c.nb * net->n[m]), dim3(kBlock),
                                     0, c.st, c.nb, t.out_c, t.out_h * t.out_w, R,
                                     m == 1 ? part1 : part2, gflag,
                                     at<int8_t>(c.ws, p.off_code) + off, c.L + off, c.U + off,
                                     net->n_relu, ga + off, gl + off, gu + off);
              }))
            return e;
        }
        continue;
      }
    }
    if (inter)  // (fused_tape_pass implies every condition of the branch above)
      return fail(LIRPA_EUNSUPPORTED, "pass %d: interleaved rows without k_fwd_conv12", P);
    // the first layer's input is the witness, built from the pass's sign tape (bytes; the
    // forward kernels with WITNESS read their input pointer as int8_t)
    const float* zin = reinterpret_cast<const float*>(tsign_of(c, P));
    float* zbuf[2] = {za, zb};
    for (int m = 1; m <= P - 1; ++m) {
      const float* tp = tape_of(c, P, m);
      long off = net->off[m], poff = net->poff[m];
      float* zout = (m < P - 1) ? zbuf[m % 2] : nullptr;
      DLayer t = dlayer(net->T[m - 1]);
      const unsigned nblk16 = (unsigned)round_up((Q + 15) / 16, 16);
      FwdKernel fk = fwd_conv_for(net->T[m - 1], m == 1, zout != nullptr);
      // fused adjoint sums (groups of 8 rows aligned to the sub-domains) where R allows it
      const bool fused = fk && P < L && R % 8 == 0 && p.off_gpart != 0;
      // an FC-opened pass recorded no tape over its first stage's input: rebuild it from W_P
      const bool wtape = m == P - 1 && fc_open_ok(c, P, R);
      const float* tapeW = wtape ? net->T[P - 1].W : nullptr;
      const int tnk = wtape ? (int)net->n[P] : 0;
      float* gpart = fused ? at<float>(c.ws, p.off_gpart) : nullptr;
      unsigned char* gflag = fused ? at<unsigned char>(c.ws, p.off_gflag) : nullptr;
      // a Linear layer past the first: the GEMM kernel (up to 128 outputs)
      const lirpa_layer& tl = net->T[m - 1];
      const bool fc_gemm = !fk && m > 1 && tl.kind == LIRPA_LINEAR && tl.in_c % 4 == 0 &&
                           tl.out_c <= 128;
      int e = launch_k(tag("fwd", m, P), c.st, [&] {
        if (fc_gemm) {
          auto kf = k_fwd_fc<8>;
          switch ((tl.out_c + 15) / 16) {
            case 1: kf = k_fwd_fc<1>; break;
            case 2: kf = k_fwd_fc<2>; break;
            case 3: kf = k_fwd_fc<3>; break;
            case 4: kf = k_fwd_fc<4>; break;
            case 5: kf = k_fwd_fc<5>; break;
            case 6: kf = k_fwd_fc<6>; break;
            case 7: kf = k_fwd_fc<7>; break;
            default: break;
          }
          const unsigned nblk64 = (unsigned)round_up((Q + 63) / 64, 8);
          hipLaunchKernelGGL(kf, dim3(nblk64), dim3(256), 0, c.st, t, zin, (unsigned)ldq,
                             (unsigned)Q, R, w, tp, at<float>(c.ws, p.off_alo) + poff,
                             at<float>(c.ws, p.off_aup) + poff, at<float>(c.ws, p.off_bup) + poff,
                             net->pstride, G, zout);
        } else if (fk) {
          // a small batch of rows (the final pass) splits each tile's output rows over two
          // blocks, so that the grid fills the GPU in whole rounds
          const int ns = (nblk16 < 4096 && t.out_h % 2 == 0) ? 2 : 1;
          hipLaunchKernelGGL(fk, dim3(nblk16 * ns), dim3(256), 0, c.st, t, zin, (unsigned)ldq,
                             (unsigned)Q, R, w, c.x0, c.eps, tp,
                             at<float>(c.ws, p.off_alo) + poff, at<float>(c.ws, p.off_aup) + poff,
                             at<float>(c.ws, p.off_bup) + poff, net->pstride, G, zout, gpart,
                             gflag, tapeW, tnk, ns);
        }
        else if (m == 1)
          hipLaunchKernelGGL(k_fwd_mfma<true>, dim3(nblk16), dim3(256), 0, c.st, t, zin,
                             (unsigned)ldq, (unsigned)Q, R, w, c.x0, c.eps, tp,
                             at<float>(c.ws, p.off_alo) + poff, at<float>(c.ws, p.off_aup) + poff,
                             at<float>(c.ws, p.off_bup) + poff, net->pstride, G, zout);
        else
          hipLaunchKernelGGL(k_fwd_mfma<false>, dim3(nblk16), dim3(256), 0, c.st, t, zin,
                             (unsigned)ldq, (unsigned)Q, R, w, c.x0, c.eps, tp,
                             at<float>(c.ws, p.off_alo) + poff, at<float>(c.ws, p.off_aup) + poff,
                             at<float>(c.ws, p.off_bup) + poff, net->pstride, G, zout);
      });
      if (e) return e;
      long pairs = c.nb * net->n[m];
      if (fused) {
        e = launch_k(tag("grad_gather", m, P), c.st, [&] {
          hipLaunchKernelGGL(k_grad_gather, grid_for(pairs), dim3(kBlock), 0, c.st, c.nb, t.out_c,
                             t.out_h * t.out_w, R, gpart, gflag,
                             at<int8_t>(c.ws, p.off_code) + off, c.L + off, c.U + off,
                             net->n_relu, ga + off, gl + off, gu + off);
        });
        if (e) return e;
        zin = zout;
        continue;
      }
      e = launch_k(tag("grad_reduce", m, P), c.st, [&] {
        if (R <= 64) {
          const long spw = R >= 4 ? 64 / R : 16;
          const long blocks = ((net->n[m] + 63) / 64) * ((c.nb + spw - 1) / spw);
          hipLaunchKernelGGL(k_grad_reduce_seg, dim3((unsigned)blocks), dim3(256),
                             0, c.st, c.nb, net->n[m], R, ldq, w, tp, G,
                             at<int8_t>(c.ws, p.off_code) + off, c.L + off, c.U + off,
                             net->n_relu, ga + off, gl + off, gu + off);
        } else {
          hipLaunchKernelGGL(k_grad_reduce, dim3((unsigned)((pairs + 3) / 4)), dim3(kBlock), 0,
                             c.st, c.nb, net->n[m], R, ldq, w, tp, G,
                             at<int8_t>(c.ws, p.off_code) + off, c.L + off, c.U + off,
                             net->n_relu, ga + off, gl + off, gu + off);
        }
      });
      if (e) return e;
      zin = zout;
    }
  }
  return LIRPA_OK;
}

int check_args(const lirpa_net* net, const float* x0, float eps, const float* C, int S, int B) {
  if (!net) return fail(LIRPA_EINVAL, "net is null");
  if (!x0) return fail(LIRPA_EINVAL, "x0 is null");
  if (!C) return fail(LIRPA_EINVAL, "C is null");
  if (S < 1) return fail(LIRPA_EINVAL, "S must be >= 1 (got %d)", S);
  if (B < 1) return fail(LIRPA_EINVAL, "B must be >= 1 (got %d)", B);
  if (!std::isfinite(eps) || eps < 0.f) return fail(LIRPA_EINVAL, "eps must be finite and >= 0");
  return LIRPA_OK;
}

int check_common(const lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                 void* ws) {
  if (int e = check_args(net, x0, eps, C, S, B)) return e;
  if (!ws) return fail(LIRPA_EINVAL, "workspace is null");
  return LIRPA_OK;
}

// Workspace plan of a call kind: 0 lirpa_bound, 1 lirpa_bound_grad / lirpa_optimize,
// 2 lirpa_bound_ul (the final pass bounds the 2S rows [C; -C]), 3 lirpa_optimize_ul (the
// optimiser's plan and the rows -C).
Plan plan_for(const lirpa_net* net, long S, long Bc, int mode) {
  if (mode <= 1) return make_plan(net, S, Bc, mode);
  Plan p = make_plan(net, mode == 2 ? 2 * S : S, Bc, mode == 2 ? 0 : 1);
  if (p.total == (size_t)-1) return p;
  const long nL = net->n[net->L];
  size_t o = p.total;
  p.off_spec = o;
  o = align256(o + (size_t)(mode == 2 ? 2 : 1) * S * nL * 4);
  if (mode == 2) {
    p.off_lb2 = o;
    o = align256(o + (size_t)Bc * 2 * S * 4);
  }
  p.total = o;
  return p;
}

// Largest chunk whose workspace fits.
long fit_chunk(const lirpa_net* net, long S, long B, size_t ws_bytes, Plan* out, int mode = 0) {
  long lo = 0, hi = B;
  while (lo < hi) {
    long mid = (lo + hi + 1) / 2;
    if (plan_for(net, S, mid, mode).total <= ws_bytes) lo = mid; else hi = mid - 1;
  }
  if (lo > 0) *out = plan_for(net, S, lo, mode);
  return lo;
}

Chunk make_chunk(lirpa_net* net, const Plan& p, void* ws, const float* x0, float eps, long S,
                 long B, long b0, const int8_t* split, const float* alpha, float* l_out,
                 float* u_out, hipStream_t stream) {
  Chunk c;
  c.net = net;
  c.p = &p;
  c.ws = ws;
  c.x0 = x0;
  c.eps = eps;
  c.S = S;
  c.nb = std::min(p.Bc, B - b0);
  c.L = l_out ? l_out + b0 * net->n_relu : at<float>(ws, p.off_l);
  c.U = u_out ? u_out + b0 * net->n_relu : at<float>(ws, p.off_u);
  c.split = split ? split + b0 * net->n_relu : nullptr;
  c.alpha = alpha ? alpha + b0 * net->n_relu : nullptr;
  c.st = stream;
  c.tape = (p.mode == 1);
  return c;
}

int copy_d2d(void* dst, const void* src, size_t bytes, hipStream_t st) {
  if (hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, st) != hipSuccess)
    return fail(LIRPA_EDEVICE, "hipMemcpyAsync failed");
  return LIRPA_OK;
}

bool validate_on() {
  const char* v = std::getenv("LIRPA_VALIDATE");
  return v && v[0] == '1' && v[1] == '\0';
}

// With LIRPA_VALIDATE=1: report (LIRPA_EDATA) and clear what the check kernels of earlier calls
// on this device found.  Synchronises the stream.
int validate_report(hipStream_t st) {
  if (!validate_on()) return LIRPA_OK;
  unsigned int f[4] = {0, 0, 0, 0};
  if (hipMemcpyFromSymbolAsync(f, HIP_SYMBOL(g_check), sizeof f, 0, hipMemcpyDeviceToHost, st) !=
          hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return fail(LIRPA_EDEVICE, "reading the input-check findings failed");
  if (!(f[0] | f[1] | f[2] | f[3])) return LIRPA_OK;
  const unsigned int zero[4] = {0, 0, 0, 0};
  if (hipMemcpyToSymbolAsync(HIP_SYMBOL(g_check), zero, sizeof zero, 0, hipMemcpyHostToDevice,
                             st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return fail(LIRPA_EDEVICE, "clearing the input-check findings failed");
  return fail(LIRPA_EDATA, "an earlier call's device inputs were out of range:%s%s%s%s",
              f[0] ? " split value outside {-1,0,1};" : "",
              f[1] ? " alpha outside [0,1];" : "", f[2] ? " non-finite x0;" : "",
              f[3] ? " non-finite C;" : "");
}

// With LIRPA_VALIDATE=1: enqueue the read-only check of this call's device inputs.
int validate_enqueue(const lirpa_net* net, const float* x0, const float* C, int S, int B,
                     const int8_t* split, const float* alpha, hipStream_t st) {
  if (!validate_on()) return LIRPA_OK;
  const long n = (long)B * net->n_relu;
  const long nC = (long)S * net->n[net->L];
  return launch_k("check_inputs", st, [&] {
    hipLaunchKernelGGL(k_check_inputs, dim3(1024), dim3(kBlock), 0, st, split ? n : 0L, split,
                       alpha ? n : 0L, alpha, net->n[0], x0, nC, C);
  });
}


// lirpa_bound on a workspace that holds chunks of Bc sub-domains (plan p).
int bound_run(lirpa_net* net, const Plan& p, long Bc, const float* x0, float eps, const float* C,
              int S, int B, const int8_t* split, const float* alpha, float* lb, float* l_out,
              float* u_out, int8_t* code_out, void* ws, hipStream_t stream,
              const float* l_par = nullptr, const float* u_par = nullptr) {
  if (int e = validate_report(stream)) return e;
  if (int e = validate_enqueue(net, x0, C, S, B, split, alpha, stream)) return e;
  if (int e = layer1_bounds(net, p, ws, x0, eps, C, S, stream)) return e;
  for (long b0 = 0; b0 < B; b0 += Bc) {
    Chunk c = make_chunk(net, p, ws, x0, eps, S, B, b0, split, alpha, l_out, u_out, stream);
    if (l_par) {
      c.lp = l_par + b0 * net->n_relu;
      c.up = u_par + b0 * net->n_relu;
    }
    if (int e = bound_chunk(c, C, lb + b0 * S)) return e;
    if (code_out && net->n_relu)
      if (int e = copy_d2d(code_out + b0 * net->n_relu, at<int8_t>(ws, p.off_code),
                           (size_t)c.nb * net->n_relu, stream))
        return e;
  }
  return LIRPA_OK;
}

constexpr int kMaxDevices = 64;
void* g_scratch_addr[kMaxDevices] = {};
std::mutex g_scratch_mu;

// The current device's copy of the scratch array, looked up once per device.
int scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0)
    return fail(LIRPA_EDEVICE, "hipGetDevice failed");
  if (dev >= kMaxDevices) return fail(LIRPA_EUNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
      return fail(LIRPA_EDEVICE, "hipGetSymbolAddress of the scratch array failed on device %d",
                  dev);
    g_scratch_addr[dev] = ptr;
  }
  *out = g_scratch_addr[dev];
  return LIRPA_OK;
}


int check_opt_params(const lirpa_opt_params& op) {
  if (op.steps < 0 || op.t0 < 0 || !(op.lr >= 0.f) || !(op.beta1 >= 0.f && op.beta1 < 1.f) ||
      !(op.beta2 >= 0.f && op.beta2 < 1.f) || !(op.eps_adam > 0.f))
    return fail(LIRPA_EINVAL, "bad optimiser parameters");
  return LIRPA_OK;
}

// lirpa_optimize on a workspace that holds chunks of Bc sub-domains (plan p, gradient mode).
int optimize_run(lirpa_net* net, const Plan& p, long Bc, const float* x0, float eps,
                 const float* C, int S, int B, const int8_t* split, float* alpha, float* adam_m,
                 float* adam_v, const lirpa_opt_params& op, float* lb_best, float* lb_trace,
                 void* ws, hipStream_t stream) {
  if (int e = layer1_bounds(net, p, ws, x0, eps, C, S, stream)) return e;
  for (long b0 = 0; b0 < B; b0 += Bc) {
    Chunk c = make_chunk(net, p, ws, x0, eps, S, B, b0, split, alpha, nullptr, nullptr, stream);
    long na = c.nb * net->n_relu, ns = c.nb * S;
    float* a = alpha + b0 * net->n_relu;
    float* lbt = at<float>(ws, p.off_lbt);
    // A fresh start bounds with the heuristic lower slopes u/(u-l) and sets alpha to them; the
    // bound at t = 0 (alpha at those values, every layer's l and u recomputed from layer 1 up)
    // then repeats that bound operation for operation.  So with steps to take, the heuristic
    // bound records the tape and serves as the t = 0 iterate.
    const bool t0_done = op.fresh && op.steps > 0;
    if (op.fresh) {
      Chunk h = c;
      h.alpha = nullptr;
      h.tape = t0_done;
      if (int e = bound_chunk(h, C, lbt)) return e;
      if (int e = launch_k("alpha_init", stream, [&] {
            hipLaunchKernelGGL(k_alpha_init, grid_for(na), dim3(kBlock), 0, stream, na, h.L, h.U,
                               a, adam_m + b0 * net->n_relu, adam_v + b0 * net->n_relu);
          }))
        return e;
    }
    const int tbase = op.fresh ? 0 : op.t0;
    for (int t = 0; t <= op.steps; ++t) {
      c.tape = (t < op.steps);
      if (!(t == 0 && t0_done))
        if (int e = bound_chunk(c, C, lbt)) return e;
      float* tr = lb_trace ? lb_trace + ((long)t * B + b0) * S : nullptr;
      if (int e = launch_k("best", stream, [&] {
            hipLaunchKernelGGL(k_best, grid_for(ns), dim3(kBlock), 0, stream, ns, lbt,
                               lb_best + b0 * S, tr, (int)(t == 0));
          }))
        return e;
      if (t == op.steps) break;
      if (int e = grad_chunk(c, 1)) return e;
      int tt = tbase + t + 1;
      float c1 = (float)(1.0 - std::pow((double)op.beta1, tt));
      float c2 = (float)(1.0 - std::pow((double)op.beta2, tt));
      if (int e = launch_k("adam", stream, [&] {
            hipLaunchKernelGGL(k_adam, grid_for(na), dim3(kBlock), 0, stream, na, a,
                               adam_m + b0 * net->n_relu, adam_v + b0 * net->n_relu,
                               at<float>(ws, p.off_ga), op.lr, op.beta1, op.beta2, op.eps_adam,
                               c1, c2);
          }))
        return e;
    }
  }
  return LIRPA_OK;
}


// lirpa_bound_ul on a workspace that holds chunks of Bc sub-domains (plan p, mode 2).
int bound_ul_run(lirpa_net* net, const Plan& p, long Bc, const float* x0, float eps,
                 const float* C, int S, int B, const int8_t* split, const float* alpha, float* lb,
                 float* ub, float* l_out, float* u_out, int8_t* code_out, void* ws,
                 hipStream_t stream) {
  const long nL = net->n[net->L];
  float* C2 = at<float>(ws, p.off_spec);
  if (int e = launch_k("spec_pm", stream, [&] {
        hipLaunchKernelGGL(k_spec_pm, grid_for((long)S * nL), dim3(kBlock), 0, stream,
                           (long)S * nL, C, C2, 1);
      }))
    return e;
  // the intermediate passes are shared; the final pass bounds the 2S rows [C; -C]
  if (int e = layer1_bounds(net, p, ws, x0, eps, C2, 2 * S, stream)) return e;
  float* lb2 = at<float>(ws, p.off_lb2);
  for (long b0 = 0; b0 < B; b0 += Bc) {
    Chunk c = make_chunk(net, p, ws, x0, eps, 2 * S, B, b0, split, alpha, l_out, u_out, stream);
    if (int e = bound_chunk(c, C2, lb2)) return e;
    if (int e = launch_k("split_ul", stream, [&] {
          hipLaunchKernelGGL(k_split_ul, grid_for(c.nb * S), dim3(kBlock), 0, stream, c.nb,
                             (long)S, lb2, lb + b0 * S, ub + b0 * S);
        }))
      return e;
    if (code_out && net->n_relu)
      if (int e = copy_d2d(code_out + b0 * net->n_relu, at<int8_t>(ws, p.off_code),
                           (size_t)c.nb * net->n_relu, stream))
        return e;
  }
  return LIRPA_OK;
}


// Branch and bound workspace: two store buffers for P, the order of P, the batch of children,
// the summary, and a region for the bounding calls on the children.
struct BabPlan {
  long cap = 0, nc = 0;  // store capacity, children per iteration (2 batch)
  bool alpha = false;     // slopes carried per record (some optimisation is asked for)
  size_t smask[2] = {}, salpha[2] = {}, slo[2] = {}, shi[2] = {}, sbr[2] = {};
  size_t perm = 0, cmask = 0, calpha = 0, cm = 0, cv = 0, clo = 0, chi = 0, clbu = 0;
  size_t cl = 0, cu = 0, ccode = 0, cbr = 0, cdst = 0, sum = 0, inner = 0;
  size_t inner_bytes = 0, total = 0;
};

BabPlan bab_plan(const lirpa_net* net, const lirpa_bab_params& bp) {
  BabPlan q;
  const long n = net->n_relu;
  q.cap = (long)bp.max_domains + bp.batch;
  q.nc = 2L * bp.batch;
  q.alpha = bp.root_steps > 0 || bp.steps > 0;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at_ = o;
    o = align256(o + bytes);
    return at_;
  };
  for (int i = 0; i < 2; ++i) {
    q.smask[i] = take((size_t)q.cap * n);
    if (q.alpha) q.salpha[i] = take((size_t)q.cap * n * 4);
    q.slo[i] = take((size_t)q.cap * 4);
    q.shi[i] = take((size_t)q.cap * 4);
    q.sbr[i] = take((size_t)q.cap * 4);
  }
  q.perm = take((size_t)q.cap * 4);
  q.cmask = take((size_t)q.nc * n);
  if (q.alpha) {
    q.calpha = take((size_t)q.nc * n * 4);
    q.cm = take((size_t)q.nc * n * 4);
    q.cv = take((size_t)q.nc * n * 4);
  }
  q.clo = take((size_t)q.nc * 4);
  q.chi = take((size_t)q.nc * 4);
  q.clbu = take((size_t)q.nc * 4);
  q.cl = take((size_t)q.nc * n * 4);
  q.cu = take((size_t)q.nc * n * 4);
  q.ccode = take((size_t)q.nc * n);
  q.cbr = take((size_t)q.nc * 4);
  q.cdst = take((size_t)q.nc * 4);
  q.sum = take(sizeof(BabSummary));
  const size_t ul = plan_for(net, 1, q.nc, 2).total;
  const size_t op = q.alpha ? plan_for(net, 1, q.nc, 1).total : 0;
  q.inner_bytes = std::max(ul, op);
  q.inner = o;
  q.total = (ul == (size_t)-1 || op == (size_t)-1) ? (size_t)-1 : o + q.inner_bytes;
  return q;
}

int check_bab_params(const lirpa_bab_params& bp) {
  if (bp.batch < 1 || bp.batch > 1024) return fail(LIRPA_EINVAL, "batch must be in 1..1024");
  if (bp.max_domains < 1 || (long)bp.max_domains + bp.batch > 16384)
    return fail(LIRPA_EINVAL, "max_domains must be >= 1 with max_domains + batch <= 16384");
  if (bp.max_iters < 0 || bp.root_steps < 0 || bp.steps < 0)
    return fail(LIRPA_EINVAL, "max_iters, root_steps and steps must be >= 0");
  if (!(bp.lr >= 0.f) || !(bp.beta1 >= 0.f && bp.beta1 < 1.f) ||
      !(bp.beta2 >= 0.f && bp.beta2 < 1.f) || !(bp.eps_adam > 0.f))
    return fail(LIRPA_EINVAL, "bad optimiser parameters");
  return LIRPA_OK;
}

// Bound nb children (masks at q.cmask, slopes at q.calpha): lower bounds into q.clo, upper
// bounds into q.chi, their l, u, codes and the neuron each would split next.  steps > 0
// optimises the slopes from where they are (fresh: from the heuristic start) first.
int bab_bound_children(lirpa_net* net, const BabPlan& q, void* ws, const float* x0, float eps,
                       const float* c, long nb, int steps, bool fresh,
                       const lirpa_bab_params& bp, hipStream_t st) {
  void* inner = at<char>(ws, q.inner);
  int8_t* mask = at<int8_t>(ws, q.cmask);
  float* alpha = q.alpha ? at<float>(ws, q.calpha) : nullptr;
  float* lo = at<float>(ws, q.clo);
  if (q.alpha && (steps > 0 || fresh)) {
    Plan p;
    const long Bc = fit_chunk(net, 1, nb, q.inner_bytes, &p, 1);
    if (Bc < 1) return fail(LIRPA_ENOMEM, "branch and bound: inner workspace too small");
    const long na = nb * net->n_relu;
    for (size_t off : {q.cm, q.cv})
      if (int e = launch_k("zero", st, [&] {
            hipLaunchKernelGGL(k_zero, grid_for(na), dim3(kBlock), 0, st, na, at<float>(ws, off));
          }))
        return e;
    lirpa_opt_params op{steps, bp.lr, bp.beta1, bp.beta2, bp.eps_adam, 0, fresh ? 1 : 0};
    if (int e = optimize_run(net, p, Bc, x0, eps, c, 1, (int)nb, mask, alpha,
                             at<float>(ws, q.cm), at<float>(ws, q.cv), op, lo, nullptr, inner,
                             st))
      return e;
  }
  // the upper bound (and l, u, codes) at the slopes the lower side ended with
  Plan p;
  const long Bc = fit_chunk(net, 1, nb, q.inner_bytes, &p, 2);
  if (Bc < 1) return fail(LIRPA_ENOMEM, "branch and bound: inner workspace too small");
  const bool opt = q.alpha && (steps > 0 || fresh);
  if (int e = bound_ul_run(net, p, Bc, x0, eps, c, 1, (int)nb, mask, alpha,
                           opt ? at<float>(ws, q.clbu) : lo, at<float>(ws, q.chi),
                           at<float>(ws, q.cl), at<float>(ws, q.cu), at<int8_t>(ws, q.ccode),
                           inner, st))
    return e;
  return launch_k("bab_branch", st, [&] {
    hipLaunchKernelGGL(k_bab_branch, dim3((unsigned)nb), dim3(kBlock), 0, st, net->n_relu,
                       at<float>(ws, q.cl), at<float>(ws, q.cu), at<int8_t>(ws, q.ccode),
                       at<int>(ws, q.cbr));
  });
}

// Domain_Filter and insertion of nc bounded children into store buffer `cur` holding N records,
// then batch_pick_out's sort of the new P; the summary is copied to *hs (the loop's one
// synchronisation per iteration).
int bab_insert_sort(lirpa_net* net, const BabPlan& q, void* ws, int cur, long N, long nc,
                    const lirpa_bab_params& bp, BabSummary* hs, hipStream_t st) {
  BabSummary* sum = at<BabSummary>(ws, q.sum);
  const long n = net->n_relu;
  if (int e = launch_k("bab_filter", st, [&] {
        hipLaunchKernelGGL(k_bab_filter, dim3(1), dim3(1024), 0, st, (int)nc, (int)N,
                           at<float>(ws, q.clo), at<float>(ws, q.chi), at<int>(ws, q.cdst), sum);
      }))
    return e;
  if (int e = launch_k("bab_insert", st, [&] {
        hipLaunchKernelGGL(k_bab_insert, grid_for(nc * n), dim3(kBlock), 0, st, nc, n,
                           at<int>(ws, q.cdst), at<int8_t>(ws, q.cmask),
                           q.alpha ? at<float>(ws, q.calpha) : nullptr, at<float>(ws, q.clo),
                           at<float>(ws, q.chi), at<int>(ws, q.cbr), at<int8_t>(ws, q.smask[cur]),
                           q.alpha ? at<float>(ws, q.salpha[cur]) : nullptr,
                           at<float>(ws, q.slo[cur]), at<float>(ws, q.shi[cur]),
                           at<int>(ws, q.sbr[cur]));
      }))
    return e;
  long npad = 1;
  while (npad < q.cap) npad <<= 1;
  const size_t lds = (size_t)npad * sizeof(unsigned long long);
  if (lds > 65536 &&
      hipFuncSetAttribute(reinterpret_cast<const void*>(k_bab_sort),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return fail(LIRPA_EDEVICE, "cannot reserve %zu bytes of LDS for the sort", lds);
  if (int e = launch_k("bab_sort", st, [&] {
        hipLaunchKernelGGL(k_bab_sort, dim3(1), dim3(1024), lds, st, bp.batch,
                           at<float>(ws, q.slo[cur]), at<float>(ws, q.shi[cur]),
                           at<int>(ws, q.sbr[cur]), at<int>(ws, q.perm), sum);
      }))
    return e;
  if (hipMemcpyAsync(hs, sum, sizeof *hs, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return fail(LIRPA_EDEVICE, "branch and bound: reading the summary failed");
  return LIRPA_OK;
}

int bab_run(lirpa_net* net, const BabPlan& q, const float* x0, float eps, const float* c,
            const lirpa_bab_params& bp, lirpa_bab_result* res, void* ws, hipStream_t st) {
  const long n = net->n_relu;
  BabSummary hs{};
  // line 2: the root (no split), optimised from the heuristic start when asked
  if (int e = launch_k("bab_init", st, [&] {
        hipLaunchKernelGGL(k_fill_i8, grid_for(n), dim3(kBlock), 0, st, n,
                           at<int8_t>(ws, q.cmask), 0);
        hipLaunchKernelGGL(k_bab_summary_init, dim3(1), dim3(1), 0, st,
                           at<BabSummary>(ws, q.sum));
      }))
    return e;
  if (int e = bab_bound_children(net, q, ws, x0, eps, c, 1, bp.root_steps, true, bp, st))
    return e;
  int cur = 0;
  long N = 0;
  // line 3: P = the root unless it is verified already
  if (int e = bab_insert_sort(net, q, ws, cur, N, 1, bp, &hs, st)) return e;
  N = hs.count;
  res->domains_bounded = 1;
  res->iterations = 0;
  for (;;) {
    int status = 0;
    if (N == 0) status = LIRPA_BAB_VERIFIED;
    else if (hs.f_hi < 0.f) status = LIRPA_BAB_VIOLATED;
    else if (N > bp.max_domains || res->iterations >= bp.max_iters) status = LIRPA_BAB_UNKNOWN_LIMIT;
    else if (hs.stuck) status = LIRPA_BAB_UNKNOWN_STUCK;
    if (status) {
      res->status = status;
      res->f_lo = N == 0 ? hs.leaf_lo : hs.f_lo;
      res->f_hi = N == 0 ? hs.leaf_hi : hs.f_hi;
      res->domains_left = (int)N;
      return LIRPA_OK;
    }
    // lines 5-6: pick the k lowest records (perm[0..k)), split each into two children; the rest
    // move to the other store buffer in order
    const long k = std::min<long>(bp.batch, N);
    if (int e = launch_k("bab_children", st, [&] {
          hipLaunchKernelGGL(k_bab_children, grid_for(2 * k * n), dim3(kBlock), 0, st, k, n,
                             at<int>(ws, q.perm), at<int8_t>(ws, q.smask[cur]),
                             q.alpha ? at<float>(ws, q.salpha[cur]) : nullptr,
                             at<int>(ws, q.sbr[cur]), at<int8_t>(ws, q.cmask),
                             q.alpha ? at<float>(ws, q.calpha) : nullptr);
        }))
      return e;
    const long rest = N - k;
    if (rest > 0)
      if (int e = launch_k("bab_gather", st, [&] {
            hipLaunchKernelGGL(k_bab_gather, grid_for(rest * n), dim3(kBlock), 0, st, rest, k, n,
                               at<int>(ws, q.perm), at<int8_t>(ws, q.smask[cur]),
                               q.alpha ? at<float>(ws, q.salpha[cur]) : nullptr,
                               at<float>(ws, q.slo[cur]), at<float>(ws, q.shi[cur]),
                               at<int>(ws, q.sbr[cur]), at<int8_t>(ws, q.smask[1 - cur]),
                               q.alpha ? at<float>(ws, q.salpha[1 - cur]) : nullptr,
                               at<float>(ws, q.slo[1 - cur]), at<float>(ws, q.shi[1 - cur]),
                               at<int>(ws, q.sbr[1 - cur]));
          }))
        return e;
    cur = 1 - cur;
    // line 7: (optimised) LiRPA on the 2k children, from their parents' slopes
    if (int e = bab_bound_children(net, q, ws, x0, eps, c, 2 * k, bp.steps, false, bp, st))
      return e;
    res->domains_bounded += 2 * k;
    // lines 8-10
    if (int e = bab_insert_sort(net, q, ws, cur, rest, 2 * k, bp, &hs, st)) return e;
    N = hs.count;
    ++res->iterations;
  }
}
}  // namespace

// ---------------------------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------------------------
extern "C" {

int lirpa_net_create(const lirpa_layer* layers, int n_layers, lirpa_net** out) {
  if (!out) return fail(LIRPA_EINVAL, "out is null");
  *out = nullptr;
  if (!layers || n_layers < 1) return fail(LIRPA_EINVAL, "need at least one layer");
  if (n_layers > kMaxLayers) return fail(LIRPA_EUNSUPPORTED, "at most %d layers", kMaxLayers);
  lirpa_net* net = new lirpa_net;
  net->L = n_layers;
  net->T.assign(layers, layers + n_layers);
  net->n[0] = n_in_of(layers[0]);
  for (int m = 1; m <= n_layers; ++m) {
    const lirpa_layer& t = layers[m - 1];
    int e = LIRPA_OK;
    if (!t.W || !t.b) e = fail(LIRPA_EINVAL, "layer %d: null W or b", m);
    else if (t.in_c < 1 || t.in_h < 1 || t.in_w < 1 || t.out_c < 1 || t.out_h < 1 || t.out_w < 1)
      e = fail(LIRPA_EINVAL, "layer %d: non-positive dimension", m);
    else if (t.kind == LIRPA_LINEAR) {
      if (t.in_h != 1 || t.in_w != 1 || t.out_h != 1 || t.out_w != 1)
        e = fail(LIRPA_EINVAL, "layer %d: a linear layer has unit spatial dims", m);
    } else if (t.kind == LIRPA_CONV2D) {
      if (t.k < 1 || t.stride < 1 || t.pad < 0)
        e = fail(LIRPA_EINVAL, "layer %d: bad conv geometry", m);
      else if (t.out_h != (t.in_h + 2 * t.pad - t.k) / t.stride + 1 ||
               t.out_w != (t.in_w + 2 * t.pad - t.k) / t.stride + 1)
        e = fail(LIRPA_EINVAL, "layer %d: conv output size does not match", m);
      else if (t.k > 7 || t.stride > 4 || t.pad >= t.k)
        e = fail(LIRPA_EUNSUPPORTED, "layer %d: conv with k<=7, stride<=4, pad<k supported", m);
    } else {
      e = fail(LIRPA_EINVAL, "layer %d: unknown kind %d", m, t.kind);
    }
    if (!e && m > 1 && n_in_of(t) != net->n[m - 1])
      e = fail(LIRPA_EINVAL, "layer %d: input size %ld != previous output size %ld", m,
               n_in_of(t), net->n[m - 1]);
    if (e) {
      delete net;
      return e;
    }
    net->n[m] = n_out_of(t);
    if (m < n_layers) {
      net->off[m] = net->n_relu;
      net->n_relu += net->n[m];
      net->poff[m] = net->pstride;
      net->pstride += round_up(net->n[m], 4);
    }
  }
  *out = net;
  return LIRPA_OK;
}

void lirpa_net_destroy(lirpa_net* net) { delete net; }

int64_t lirpa_net_num_relu(const lirpa_net* net) { return net ? net->n_relu : -1; }

size_t lirpa_workspace_bytes(const lirpa_net* net, int S, int B_chunk, int mode) {
  if (!net || S < 1 || B_chunk < 1 || mode < 0 || mode > 3) return 0;
  return plan_for(net, S, B_chunk, mode).total;
}

int lirpa_bound(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                const int8_t* split, const float* alpha, float* lb, float* l_out, float* u_out,
                int8_t* code_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (int e = check_common(net, x0, eps, C, S, B, ws)) return e;
  if (!lb) return fail(LIRPA_EINVAL, "lb is null");
  if ((l_out == nullptr) != (u_out == nullptr))
    return fail(LIRPA_EINVAL, "l_out and u_out must both be given or both be null");
  Plan p;
  long Bc = fit_chunk(net, S, B, ws_bytes, &p);
  if (Bc < 1)
    return fail(LIRPA_ENOMEM, "workspace of %zu bytes holds no sub-domain (need %zu)", ws_bytes,
                make_plan(net, S, 1).total);
  return bound_run(net, p, Bc, x0, eps, C, S, B, split, alpha, lb, l_out, u_out, code_out, ws,
                   stream);
}

int lirpa_bound_child(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                      const int8_t* split, const float* alpha, const float* l_parent,
                      const float* u_parent, float* lb, float* l_out, float* u_out,
                      int8_t* code_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (int e = check_common(net, x0, eps, C, S, B, ws)) return e;
  if (!lb) return fail(LIRPA_EINVAL, "lb is null");
  if (!l_parent || !u_parent) return fail(LIRPA_EINVAL, "l_parent and u_parent must be given");
  if ((l_out == nullptr) != (u_out == nullptr))
    return fail(LIRPA_EINVAL, "l_out and u_out must both be given or both be null");
  Plan p;
  long Bc = fit_chunk(net, S, B, ws_bytes, &p);
  if (Bc < 1)
    return fail(LIRPA_ENOMEM, "workspace of %zu bytes holds no sub-domain (need %zu)", ws_bytes,
                make_plan(net, S, 1).total);
  return bound_run(net, p, Bc, x0, eps, C, S, B, split, alpha, lb, l_out, u_out, code_out, ws,
                   stream, l_parent, u_parent);
}

int lirpa_bound_noalloc(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                        const int8_t* split, const float* alpha, float* lb, float* l_out,
                        float* u_out, int8_t* code_out, hipStream_t stream) {
  // host checks first: a rejected call touches no device
  if (int e = check_args(net, x0, eps, C, S, B)) return e;
  if (!lb) return fail(LIRPA_EINVAL, "lb is null");
  if ((l_out == nullptr) != (u_out == nullptr))
    return fail(LIRPA_EINVAL, "l_out and u_out must both be given or both be null");
  Plan p;
  long Bc = fit_chunk(net, S, B, kScratchBytes, &p);
  if (Bc < 1)
    return fail(LIRPA_ENOMEM,
                "one sub-domain needs %zu bytes of workspace, beyond the library's scratch array "
                "of %zu MiB; call lirpa_bound with a workspace",
                make_plan(net, S, 1).total, kScratchBytes >> 20);
  void* ws = nullptr;
  if (int e = scratch_address(&ws)) return e;
  return bound_run(net, p, Bc, x0, eps, C, S, B, split, alpha, lb, l_out, u_out, code_out, ws,
                   stream);
}

int lirpa_bound_grad(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                     const int8_t* split, const float* alpha, int full, float* lb, float* grad,
                     void* ws, size_t ws_bytes, hipStream_t stream) {
  if (int e = check_common(net, x0, eps, C, S, B, ws)) return e;
  if (!alpha) return fail(LIRPA_EINVAL, "alpha is required for the gradient");
  if (!lb || !grad) return fail(LIRPA_EINVAL, "lb and grad must be given");
  Plan p;
  long Bc = fit_chunk(net, S, B, ws_bytes, &p, 1);
  if (Bc < 1)
    return fail(LIRPA_ENOMEM, "workspace of %zu bytes holds no sub-domain (need %zu)", ws_bytes,
                make_plan(net, S, 1, 1).total);
  if (int e = validate_report(stream)) return e;
  if (int e = validate_enqueue(net, x0, C, S, B, split, alpha, stream)) return e;
  if (int e = layer1_bounds(net, p, ws, x0, eps, C, S, stream)) return e;
  for (long b0 = 0; b0 < B; b0 += Bc) {
    Chunk c = make_chunk(net, p, ws, x0, eps, S, B, b0, split, alpha, nullptr, nullptr, stream);
    if (int e = bound_chunk(c, C, lb + b0 * S)) return e;
    if (int e = grad_chunk(c, full)) return e;
    if (int e = copy_d2d(grad + b0 * net->n_relu, at<float>(ws, p.off_ga),
                         sizeof(float) * c.nb * net->n_relu, stream))
      return e;
  }
  return LIRPA_OK;
}

int lirpa_optimize(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                   const int8_t* split, float* alpha, float* adam_m, float* adam_v,
                   const lirpa_opt_params* params, float* lb_best, float* lb_trace, void* ws,
                   size_t ws_bytes, hipStream_t stream) {
  if (int e = check_common(net, x0, eps, C, S, B, ws)) return e;
  if (!alpha || !adam_m || !adam_v || !params || !lb_best)
    return fail(LIRPA_EINVAL, "alpha, adam_m, adam_v, params and lb_best must be given");
  if (int e = check_opt_params(*params)) return e;
  Plan p;
  long Bc = fit_chunk(net, S, B, ws_bytes, &p, 1);
  if (Bc < 1)
    return fail(LIRPA_ENOMEM, "workspace of %zu bytes holds no sub-domain (need %zu)", ws_bytes,
                make_plan(net, S, 1, 1).total);
  if (int e = validate_report(stream)) return e;
  // alpha is an input only when the call continues from the caller's state
  if (int e = validate_enqueue(net, x0, C, S, B, split, params->fresh ? nullptr : alpha, stream))
    return e;
  return optimize_run(net, p, Bc, x0, eps, C, S, B, split, alpha, adam_m, adam_v, *params,
                      lb_best, lb_trace, ws, stream);
}

int lirpa_bound_ul(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                   const int8_t* split, const float* alpha, float* lb, float* ub, float* l_out,
                   float* u_out, int8_t* code_out, void* ws, size_t ws_bytes,
                   hipStream_t stream) {
  if (int e = check_common(net, x0, eps, C, S, B, ws)) return e;
  if (!lb || !ub) return fail(LIRPA_EINVAL, "lb and ub must be given");
  if ((l_out == nullptr) != (u_out == nullptr))
    return fail(LIRPA_EINVAL, "l_out and u_out must both be given or both be null");
  Plan p;
  long Bc = fit_chunk(net, S, B, ws_bytes, &p, 2);
  if (Bc < 1)
    return fail(LIRPA_ENOMEM, "workspace of %zu bytes holds no sub-domain (need %zu)", ws_bytes,
                plan_for(net, S, 1, 2).total);
  if (int e = validate_report(stream)) return e;
  if (int e = validate_enqueue(net, x0, C, S, B, split, alpha, stream)) return e;
  return bound_ul_run(net, p, Bc, x0, eps, C, S, B, split, alpha, lb, ub, l_out, u_out, code_out,
                      ws, stream);
}

int lirpa_optimize_ul(lirpa_net* net, const float* x0, float eps, const float* C, int S, int B,
                      const int8_t* split, float* alpha_lo, float* m_lo, float* v_lo,
                      float* alpha_up, float* m_up, float* v_up, const lirpa_opt_params* params,
                      float* lb_best, float* ub_best, void* ws, size_t ws_bytes,
                      hipStream_t stream) {
  if (int e = check_common(net, x0, eps, C, S, B, ws)) return e;
  if (!alpha_lo || !m_lo || !v_lo || !alpha_up || !m_up || !v_up || !params || !lb_best ||
      !ub_best)
    return fail(LIRPA_EINVAL, "both sides' alpha, m, v, params, lb_best and ub_best must be given");
  if (int e = check_opt_params(*params)) return e;
  Plan p;
  long Bc = fit_chunk(net, S, B, ws_bytes, &p, 3);
  if (Bc < 1)
    return fail(LIRPA_ENOMEM, "workspace of %zu bytes holds no sub-domain (need %zu)", ws_bytes,
                plan_for(net, S, 1, 3).total);
  if (int e = validate_report(stream)) return e;
  if (int e = validate_enqueue(net, x0, C, S, B, split, params->fresh ? nullptr : alpha_lo,
                               stream))
    return e;
  if (!params->fresh)
    if (int e = validate_enqueue(net, x0, C, S, B, nullptr, alpha_up, stream)) return e;
  // lower side: maximise lb of C over alpha_lo
  if (int e = optimize_run(net, p, Bc, x0, eps, C, S, B, split, alpha_lo, m_lo, v_lo, *params,
                           lb_best, nullptr, ws, stream))
    return e;
  // upper side: maximise lb of -C over alpha_up, i.e. minimise ub = -lb(-C) (Eq. 9 read as the
  // tightest sound upper bound)
  const long nL = net->n[net->L];
  float* Cn = at<float>(ws, p.off_spec);
  if (int e = launch_k("spec_pm", stream, [&] {
        hipLaunchKernelGGL(k_spec_pm, grid_for((long)S * nL), dim3(kBlock), 0, stream,
                           (long)S * nL, C, Cn, 0);
      }))
    return e;
  if (int e = optimize_run(net, p, Bc, x0, eps, Cn, S, B, split, alpha_up, m_up, v_up, *params,
                           ub_best, nullptr, ws, stream))
    return e;
  return launch_k("negate", stream, [&] {
    hipLaunchKernelGGL(k_negate, grid_for((long)B * S), dim3(kBlock), 0, stream, (long)B * S,
                       ub_best);
  });
}

size_t lirpa_bab_workspace_bytes(const lirpa_net* net, const lirpa_bab_params* params) {
  if (!net || !params || check_bab_params(*params)) return 0;
  return bab_plan(net, *params).total;
}

int lirpa_bab(lirpa_net* net, const float* x0, float eps, const float* c,
              const lirpa_bab_params* params, lirpa_bab_result* result, void* ws,
              size_t ws_bytes, hipStream_t stream) {
  if (int e = check_common(net, x0, eps, c, 1, 1, ws)) return e;
  if (!params || !result) return fail(LIRPA_EINVAL, "params and result must be given");
  if (int e = check_bab_params(*params)) return e;
  const BabPlan q = bab_plan(net, *params);
  if (q.total > ws_bytes)
    return fail(LIRPA_ENOMEM, "workspace of %zu bytes, branch and bound needs %zu", ws_bytes,
                q.total);
  if (int e = validate_report(stream)) return e;
  if (int e = validate_enqueue(net, x0, c, 1, 1, nullptr, nullptr, stream)) return e;
  *result = lirpa_bab_result{};
  return bab_run(net, q, x0, eps, c, *params, result, ws, stream);
}

int lirpa_timing_begin(void) {
  g_tim.on = true;
  g_tim.used = 0;
  g_tim.recs.clear();
  return LIRPA_OK;
}

int lirpa_timing_end(lirpa_kernel_time* out, int max_entries, int* n) {
  g_tim.on = false;
  std::vector<lirpa_kernel_time> acc;
  int rc = LIRPA_OK;
  for (const TimingRec& r : g_tim.recs) {
    float ms = 0.f;
    if (hipEventSynchronize(g_tim.pool[r.ev + 1]) != hipSuccess ||
        hipEventElapsedTime(&ms, g_tim.pool[r.ev], g_tim.pool[r.ev + 1]) != hipSuccess) {
      rc = fail(LIRPA_EDEVICE, "timing events failed");
      break;
    }
    auto it = std::find_if(acc.begin(), acc.end(),
                           [&](const lirpa_kernel_time& k) { return r.cls == k.name; });
    if (it == acc.end()) {
      lirpa_kernel_time k{};
      snprintf(k.name, sizeof k.name, "%s", r.cls.c_str());
      acc.push_back(k);
      it = acc.end() - 1;
    }
    it->total_ms += ms;
    it->launches += 1;
  }
  g_tim.recs.clear();
  g_tim.used = 0;
  if (n) *n = (int)acc.size();
  for (int i = 0; out && i < (int)acc.size() && i < max_entries; ++i) out[i] = acc[i];
  return rc;
}

const char* lirpa_last_error(void) { return g_err.c_str(); }

}  // extern "C"
