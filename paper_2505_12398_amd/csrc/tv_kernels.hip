// Traversal Verification (arXiv 2505.12398, Algorithm 3) and the token-level
// baseline (Sec. 2.2, Algorithm 2 per node) for gfx950 (MI355X, CDNA4).
//
// One 1024-thread workgroup verifies one tree. Thread 0 runs the sequential
// traversal on scalars held in LDS and issues vocabulary-wide passes that all
// 16 wavefronts execute over the rows of one node, 16 bytes per lane per load:
//
//   STATS   row maxima and sums of 2^(z*k - m*k) (k = log2(e)/T) for the target
//           and draft rows of a node, plus the parent's logits at each child's
//           token; run lazily, the first time the traversal descends into a
//           node whose acceptance rate is above zero;
//   SPASS   S = sum_x [alpha p(x) - beta q(x)]_+, one per rejection: Eq. (e1)
//           and (e3) for the rejected node's parent;
//   SAMPLE  inverse-CDF draw of Y from [A p - B q]_+ (or the target row of an
//           accepted leaf), in ascending token order.
//
// A node's residual target and draft are never materialised: after k
// rejections they are b = [A p - B q]_+ and s = c q off the rejected tokens,
// so four scalars (pi, A, B, rejected draft mass) carry Eq. (e1)-(e3) and a
// sibling's ratio b/s = [A r - B]_+ / c needs no vocabulary pass. The literal
// vector form of Algorithm 3 and this four-scalar form give the same values
// (the CPU tests check it); the traversal order, tests and outputs are those of
// Algorithm 3.
//
// Precision. Logits are widened exactly to fp32 and every per-node scalar is
// fp64. Two element paths: FAST (bf16 logits with V >= 16384) takes each term
// as the hardware exp2 of an fp32 fma and combines and accumulates in fp64;
// over a large vocabulary the per-element rounding averages out. PRECISE (fp32
// logits, or any V < 16384) evaluates every term with fp64 exp2. In both, the
// remaining draft mass 1 - q(rejected tokens) comes from the pass's own sum of
// draft terms minus the rejected tokens' terms (recomputed bit-identically),
// never from 1 - sum q, which cancels when the rejected tokens held most of the
// draft mass.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tv.h"
#include "tv_launch.h"

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxNodes = TV_MAX_NODES;
constexpr int kMaxBlocks = 2048;   // sampling blocks (64 * bmul vectors each)
constexpr int kUnroll = 4;         // vectors per row in flight per lane

enum : int { kCmdDone = 0, kCmdStats = 1, kCmdSPass = 2, kCmdSample = 3 };
enum : int {
  kPhDescend = 0, kPhTest, kPhAfterSPass, kPhFinal, kPhFinalLeafStats, kPhAfterSample,
  kPhPinit, kPhTlVisit, kPhTlAfterSPass
};
enum : uint8_t { kFlagStats = 1, kFlagConsulted = 2, kFlagLeafStats = 4, kFlagSd = 8 };

struct TreeSmem {
  // tree structure
  int16_t parent[kMaxNodes];
  int16_t depth[kMaxNodes];
  int16_t child_start[kMaxNodes];
  int16_t child_list[kMaxNodes];
  int16_t next_child[kMaxNodes];     // children already removed (always a prefix)
  int32_t child_count[kMaxNodes];
  int32_t token[kMaxNodes];
  float u[kMaxNodes];
  uint8_t state[kMaxNodes];
  uint8_t flags[kMaxNodes];
  float theta[kMaxNodes];
  // per-node verification state
  double pi[kMaxNodes];              // current acceptance rate p of the chain ending here
  double A[kMaxNodes];               // residual target b = [A p - B q]_+
  double B[kMaxNodes];
  double rem[kMaxNodes];             // draft mass left after removing rejected tokens
  double pini[kMaxNodes];
  double sdsum[kMaxNodes];           // sum of the draft row's terms in its frame
  double invsb[kMaxNodes];           // 1 / (sum of the target row's terms)
  double invss[kMaxNodes];           // 1 / (sum of the draft row's terms)
  double cb[kMaxNodes];              // exponent offset of the target row: -max * k
  double cs[kMaxNodes];              // exponent offset of the draft row
  // per-node, about the node's own token at its parent (set by the parent's STATS)
  double r0[kMaxNodes];              // original ratio p(x) / q(x)
  double et[kMaxNodes];              // draft term of x in the parent's frame
  // sampling
  double blocks[kMaxBlocks];
  // reductions
  double red_d[2 * kWaves];
  float red_f[2 * kWaves];
  int gather_bad;
  // command issued by thread 0 for the whole workgroup
  int cmd, cmd_node, cmd_two_rows, cmd_gather, cmd_sd;
  double cmd_ap, cmd_bp;             // multipliers of the target / draft terms
  double cmd_cb, cmd_cs;
  // pass results
  float res_m[2];
  double res_s[2];
  double res_S;
  double res_sd;                     // sum of the draft terms of the last SPASS
  double res_head, res_tail;
  int res_y;
  int res_block;
  int res_bad;
  // traversal state
  int phase, cur, accepted, rejected, status, algo;
  int rows_consulted, resid_passes, tests, pinit_next;
  double alpha, beta;
};

// ---------------------------------------------------------------------------
// Element access
// ---------------------------------------------------------------------------

template <typename T> struct Elem;

template <> struct Elem<uint16_t> {          // bfloat16 bit patterns
  static constexpr int E = 8;
  __device__ static inline void unpack(const uint4& v, float (&x)[8]) {
    x[0] = __uint_as_float(v.x << 16); x[1] = __uint_as_float(v.x & 0xffff0000u);
    x[2] = __uint_as_float(v.y << 16); x[3] = __uint_as_float(v.y & 0xffff0000u);
    x[4] = __uint_as_float(v.z << 16); x[5] = __uint_as_float(v.z & 0xffff0000u);
    x[6] = __uint_as_float(v.w << 16); x[7] = __uint_as_float(v.w & 0xffff0000u);
  }
  __device__ static inline float scalar(const uint16_t* p) {
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
  }
};

template <> struct Elem<float> {
  static constexpr int E = 4;
  __device__ static inline void unpack(const uint4& v, float (&x)[4]) {
    x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y);
    x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
  }
  __device__ static inline float scalar(const float* p) { return *p; }
};

// A row split into a scalar head (up to the first 16-byte boundary), full
// 16-byte vectors, and a scalar tail. Target and draft rows of a node share
// the same split (the host checks the two tensors agree modulo 16 bytes).
struct Geom {
  int head, nvec, tail;
};

template <typename T>
__device__ inline Geom row_geom(const T* row, int V) {
  constexpr int E = Elem<T>::E;
  const int mis = static_cast<int>(reinterpret_cast<uintptr_t>(row) & 15);
  int head = mis ? (16 - mis) / static_cast<int>(sizeof(T)) : 0;
  head = head < V ? head : V;
  const int rest = V - head;
  return Geom{head, rest / E, rest % E};
}

template <typename T>
__device__ inline uint4 load16(const T* row, int head, int v) {
  return *reinterpret_cast<const uint4*>(row + head + v * Elem<T>::E);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------------------
// Workgroup reductions (fixed order: deterministic)
// ---------------------------------------------------------------------------

__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Sums of two doubles per thread in one LDS round; results valid in every thread.
__device__ __forceinline__ void block_sum2(TreeSmem& sm, double& a, double& b) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  a = wave_sum(a);
  b = wave_sum(b);
  if (lane == 0) {
    sm.red_d[wave] = a;
    sm.red_d[kWaves + wave] = b;
  }
  __syncthreads();
  double ta = 0.0, tb = 0.0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    ta += sm.red_d[w];
    tb += sm.red_d[kWaves + w];
  }
  __syncthreads();
  a = ta;
  b = tb;
}

__device__ __forceinline__ void block_max2(TreeSmem& sm, float& a, float& b) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  a = wave_max(a);
  b = wave_max(b);
  if (lane == 0) {
    sm.red_f[wave] = a;
    sm.red_f[kWaves + wave] = b;
  }
  __syncthreads();
  float ta = -INFINITY, tb = -INFINITY;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    ta = fmaxf(ta, sm.red_f[w]);
    tb = fmaxf(tb, sm.red_f[kWaves + w]);
  }
  __syncthreads();
  a = ta;
  b = tb;
}

// ---------------------------------------------------------------------------
// Element arithmetic. A row's terms are 2^(z*k + c) for a frame offset c
// (c = -max * k once the row maximum is known).
// ---------------------------------------------------------------------------

struct FastArith {                 // hardware exp2 of an fp32 fma
  static constexpr bool kPrecise = false;
  float k;                         // log2(e) / T rounded to fp32
  __device__ double frame(float m) const { return static_cast<double>(-m * k); }
  __device__ double ex(float z, double c) const {
    return static_cast<double>(fast_exp2(fmaf(z, k, static_cast<float>(c))));
  }
  __device__ double kd() const { return static_cast<double>(k); }
};

struct PreciseArith {              // fp64 throughout
  static constexpr bool kPrecise = true;
  double k;                        // log2(e) / T
  __device__ double frame(float m) const { return -static_cast<double>(m) * k; }
  __device__ double ex(float z, double c) const {
    return exp2(fma(static_cast<double>(z), k, c));
  }
  __device__ double kd() const { return k; }
};

// ---------------------------------------------------------------------------
// STATS: row maximum and sum of terms, online over one read of the row
// ---------------------------------------------------------------------------

// Running state of one thread over a row. Before the first finite value the
// maximum is -inf and the frame is that of a finite sentinel, so -inf entries
// add 2^-inf = 0 with no branch, a NaN or +inf entry turns the sum into NaN,
// and a row with no finite entry keeps maximum -inf.
constexpr float kFrameSentinel = -1.0e30f;

struct Online {
  float m;     // running max
  double c;    // frame of m (of the sentinel while m = -inf)
  double s;    // sum of terms in the frame c
};

template <class A>
__device__ __forceinline__ Online online_init(const A& ar) {
  return Online{-INFINITY, ar.frame(kFrameSentinel), 0.0};
}

// Raise the running maximum to at least vmax (rescaling the sum), then add the
// terms of x[0..n).
template <class A>
__device__ __forceinline__ void online_raise(Online& o, float vmax, const A& ar) {
  if (vmax > o.m) {
    const double cn = ar.frame(vmax);
    if constexpr (A::kPrecise) {
      o.s *= exp2(cn - o.c);
    } else {        // fp32 rescale: ~1e-7 relative, random across threads
      o.s *= static_cast<double>(fast_exp2(static_cast<float>(cn - o.c)));
    }
    o.m = vmax;
    o.c = cn;
  }
}

template <class A, int N>
__device__ __forceinline__ void online_sum(Online& o, const float (&x)[N], const A& ar) {
  if constexpr (A::kPrecise) {
#pragma unroll
    for (int e = 0; e < N; ++e) o.s += ar.ex(x[e], o.c);
  } else {
    const float cf = static_cast<float>(o.c);
    float part = 0.0f;
#pragma unroll
    for (int e = 0; e < N; ++e) part += fast_exp2(fmaf(x[e], ar.k, cf));
    o.s += static_cast<double>(part);
  }
}

template <int N>
__device__ __forceinline__ float vec_max(const float (&x)[N]) {
  float m = x[0];
#pragma unroll
  for (int e = 1; e < N; ++e) m = fmaxf(m, x[e]);
  return m;
}

template <typename T, class A, bool TWO>
__device__ __forceinline__ void stats_pass(TreeSmem& sm, const T* rb, const T* rs, int V,
                                           const A& ar, int node, bool gather) {
  constexpr int E = Elem<T>::E;
  const int tid = threadIdx.x;
  // The parent's logits at its children's tokens: loaded now, used after the
  // reduction (by the same threads), so the row stream does not wait on them.
  const bool gthread = gather && tid < sm.child_count[node];
  int gchild = 0;
  float gb = 0.0f, gs = 0.0f;
  if (gthread) {
    gchild = sm.child_list[sm.child_start[node] + tid];
    const int x = sm.token[gchild];
    gb = Elem<T>::scalar(rb + x);
    gs = Elem<T>::scalar(rs + x);
  }
  const Geom g = row_geom(rb, V);
  Online ob = online_init(ar), os = online_init(ar);
  auto scalar_elem = [&](int i) {
    float xb[1] = {Elem<T>::scalar(rb + i)};
    online_raise(ob, xb[0], ar);
    online_sum(ob, xb, ar);
    if constexpr (TWO) {
      float xs[1] = {Elem<T>::scalar(rs + i)};
      online_raise(os, xs[0], ar);
      online_sum(os, xs, ar);
    }
  };
  if (tid < g.head) scalar_elem(tid);
  if (tid < g.tail) scalar_elem(g.head + g.nvec * E + tid);
  for (int v0 = tid; v0 < g.nvec; v0 += kThreads * kUnroll) {
    uint4 lb[kUnroll], ls[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int v = v0 + u * kThreads;
      if (v < g.nvec) {
        lb[u] = load16(rb, g.head, v);
        if constexpr (TWO) ls[u] = load16(rs, g.head, v);
      }
    }
    // one rescale per group of kUnroll vectors and row
    float xb[kUnroll][E], xs[kUnroll][E];
    float mb = -INFINITY, ms = -INFINITY;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (v0 + u * kThreads < g.nvec) {
        Elem<T>::unpack(lb[u], xb[u]);
        mb = fmaxf(mb, vec_max(xb[u]));
        if constexpr (TWO) {
          Elem<T>::unpack(ls[u], xs[u]);
          ms = fmaxf(ms, vec_max(xs[u]));
        }
      }
    }
    online_raise(ob, mb, ar);
    if constexpr (TWO) online_raise(os, ms, ar);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (v0 + u * kThreads < g.nvec) {
        online_sum(ob, xb[u], ar);
        if constexpr (TWO) online_sum(os, xs[u], ar);
      }
    }
  }
  // both rows' maxima in one round, then both rows' sums in one round
  float Mb = ob.m, Ms = TWO ? os.m : -INFINITY;
  block_max2(sm, Mb, Ms);
  const double Cb = ar.frame(Mb);
  const double Cs = TWO ? ar.frame(Ms) : 0.0;
  // exact fp64 change of frame; a thread that saw no finite value has s = 0
  // (or NaN) and a factor 0 unless the whole row has no finite value
  double Sb = ob.s * exp2(Cb - ob.c);
  double Ss = TWO ? os.s * exp2(Cs - os.c) : 0.0;
  block_sum2(sm, Sb, Ss);
  const bool bad = !(Mb > -INFINITY) || !isfinite(Sb) ||
                   (TWO && (!(Ms > -INFINITY) || !isfinite(Ss)));
  if (tid == 0) {
    sm.cb[node] = Cb;
    sm.invsb[node] = 1.0 / Sb;
    if constexpr (TWO) {
      sm.cs[node] = Cs;
      sm.invss[node] = 1.0 / Ss;
    }
    sm.res_bad = bad ? 1 : 0;
    sm.gather_bad = 0;
  }
  __syncthreads();
  // Children's original ratios r0 = p(x)/q(x) and draft terms, one thread each.
  if (gthread && !bad) {
    const double kd = ar.kd();
    const double lp = fma(static_cast<double>(gb), kd, Cb) - log2(Sb);
    const double lq = fma(static_cast<double>(gs), kd, Cs) - log2(Ss);
    sm.r0[gchild] = exp2(lp - lq);
    sm.et[gchild] = ar.ex(gs, Cs);
    if (gs == -INFINITY) sm.gather_bad = 1;     // token the draft cannot produce
  }
  __syncthreads();
  if (tid == 0 && sm.gather_bad) sm.res_bad = 1;
}

// ---------------------------------------------------------------------------
// Residual weights max(ap * tb - bp * ts, 0), tb and ts the target and draft
// terms of an element (TWO == false: target only, weight ap * tb). With SD the
// draft terms are also summed, exactly in fp64.
// ---------------------------------------------------------------------------

struct TermParams {
  double cb, cs;   // frames of the target and draft rows
  double ap, bp;   // multipliers of the target and draft terms
};

template <class A, bool TWO, bool SD> struct Terms;

// Fast path: fp32 per element; the weights of one vector are summed in fp32
// and the vector sums in fp64.
template <bool TWO, bool SD> struct Terms<FastArith, TWO, SD> {
  float k, cb, cs, ap, bp;
  __device__ Terms(const FastArith& ar, const TermParams& p)
      : k(ar.k), cb(static_cast<float>(p.cb)), cs(static_cast<float>(p.cs)),
        ap(static_cast<float>(p.ap)), bp(static_cast<float>(p.bp)) {}
  template <int N>
  __device__ __forceinline__ void weights(const float (&zb)[N], const float (&zs)[N],
                                          float (&w)[N], double& sd) const {
#pragma unroll
    for (int e = 0; e < N; ++e) {
      const float eb = fast_exp2(fmaf(zb[e], k, cb));
      if constexpr (TWO) {
        const float es = fast_exp2(fmaf(zs[e], k, cs));
        if constexpr (SD) sd += static_cast<double>(es);
        w[e] = fmaxf(fmaf(eb, ap, -es * bp), 0.0f);
      } else {
        w[e] = eb * ap;
      }
    }
  }
  template <int N>
  __device__ __forceinline__ double sum(const float (&zb)[N], const float (&zs)[N],
                                        double& sd) const {
    float w[N];
    weights(zb, zs, w, sd);
    float acc = 0.0f;
#pragma unroll
    for (int e = 0; e < N; ++e) acc += w[e];
    return static_cast<double>(acc);
  }
};

// Precise path: fp64 throughout.
template <bool TWO, bool SD> struct Terms<PreciseArith, TWO, SD> {
  double k, cb, cs, ap, bp;
  __device__ Terms(const PreciseArith& ar, const TermParams& p)
      : k(ar.k), cb(p.cb), cs(p.cs), ap(p.ap), bp(p.bp) {}
  template <int N>
  __device__ __forceinline__ void weights(const float (&zb)[N], const float (&zs)[N],
                                          double (&w)[N], double& sd) const {
#pragma unroll
    for (int e = 0; e < N; ++e) {
      const double eb = exp2(fma(static_cast<double>(zb[e]), k, cb));
      if constexpr (TWO) {
        const double es = exp2(fma(static_cast<double>(zs[e]), k, cs));
        if constexpr (SD) sd += es;
        w[e] = fmax(fma(eb, ap, -es * bp), 0.0);
      } else {
        w[e] = eb * ap;
      }
    }
  }
  template <int N>
  __device__ __forceinline__ double sum(const float (&zb)[N], const float (&zs)[N],
                                        double& sd) const {
    double w[N];
    weights(zb, zs, w, sd);
    double acc = 0.0;
#pragma unroll
    for (int e = 0; e < N; ++e) acc += w[e];
    return acc;
  }
};

template <typename T, class TM, bool TWO>
__device__ __forceinline__ double vec_sum(const TM& tm, const uint4& vb, const uint4& vs,
                                          double& sd) {
  constexpr int E = Elem<T>::E;
  float xb[E], xs[E];
  Elem<T>::unpack(vb, xb);
  if constexpr (TWO) Elem<T>::unpack(vs, xs);
  else {
#pragma unroll
    for (int e = 0; e < E; ++e) xs[e] = 0.0f;
  }
  return tm.sum(xb, xs, sd);
}

template <typename T, class TM, bool TWO>
__device__ __forceinline__ double scalar_weight(const TM& tm, const T* rb, const T* rs, int i,
                                                double& sd) {
  float xb[1] = {Elem<T>::scalar(rb + i)};
  float xs[1] = {TWO ? Elem<T>::scalar(rs + i) : 0.0f};
  return tm.sum(xb, xs, sd);
}

// S = sum of the residual weights (Eq. e1, e3); with SD also the draft-term sum.
template <typename T, class A, bool SD>
__device__ __forceinline__ void s_pass(TreeSmem& sm, const T* rb, const T* rs, int V,
                                       const A& ar, const TermParams& p) {
  const Terms<A, true, SD> tm(ar, p);
  const int tid = threadIdx.x;
  const Geom g = row_geom(rb, V);
  double acc = 0.0, sd = 0.0;
  if (tid < g.head) acc += scalar_weight<T, decltype(tm), true>(tm, rb, rs, tid, sd);
  const int tail0 = g.head + g.nvec * Elem<T>::E;
  if (tid < g.tail) acc += scalar_weight<T, decltype(tm), true>(tm, rb, rs, tail0 + tid, sd);
  for (int v0 = tid; v0 < g.nvec; v0 += kThreads * kUnroll) {
    uint4 lb[kUnroll], ls[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int v = v0 + u * kThreads;
      if (v < g.nvec) {
        lb[u] = load16(rb, g.head, v);
        ls[u] = load16(rs, g.head, v);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int v = v0 + u * kThreads;
      if (v < g.nvec) acc += vec_sum<T, decltype(tm), true>(tm, lb[u], ls[u], sd);
    }
  }
  block_sum2(sm, acc, sd);
  if (tid == 0) {
    sm.res_S = acc;
    if constexpr (SD) sm.res_sd = sd;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// SAMPLE: inverse CDF over the residual weights, ascending token order.
// Order of the running sum: head elements, then blocks of 64 vectors (one per
// wavefront and iteration), then tail elements.
// ---------------------------------------------------------------------------

template <typename T, class A, bool TWO>
__device__ __forceinline__ void sample_pass(TreeSmem& sm, const T* rb, const T* rs, int V,
                                            const A& ar, const TermParams& p, float u) {
  constexpr int E = Elem<T>::E;
  constexpr int kU = 2;            // iterations (vectors per lane) in flight
  const Terms<A, TWO, false> tm(ar, p);
  using TM = Terms<A, TWO, false>;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const Geom g = row_geom(rb, V);
  const int tail0 = g.head + g.nvec * E;
  const int nblocks = (g.nvec + 63) / 64;
  const int iters = (g.nvec + kThreads - 1) / kThreads;
  double unused = 0.0;
  for (int it0 = 0; it0 < iters; it0 += kU) {
    uint4 lb[kU], ls[kU];
#pragma unroll
    for (int q = 0; q < kU; ++q) {
      const int v = (it0 + q) * kThreads + tid;
      lb[q] = make_uint4(0, 0, 0, 0);
      ls[q] = make_uint4(0, 0, 0, 0);
      if (v < g.nvec) {
        lb[q] = load16(rb, g.head, v);
        if constexpr (TWO) ls[q] = load16(rs, g.head, v);
      }
    }
#pragma unroll
    for (int q = 0; q < kU; ++q) {
      if (it0 + q < iters) {
        const int v = (it0 + q) * kThreads + tid;
        double l = v < g.nvec ? vec_sum<T, TM, TWO>(tm, lb[q], ls[q], unused) : 0.0;
        l = wave_sum(l);
        const int blk = (it0 + q) * kWaves + wave;
        if (lane == 0 && blk < nblocks) sm.blocks[blk] = l;
      }
    }
  }
  if (tid == 0) {
    double h = 0.0, tl = 0.0;
    for (int i = 0; i < g.head; ++i) h += scalar_weight<T, TM, TWO>(tm, rb, rs, i, unused);
    for (int i = tail0; i < V; ++i) tl += scalar_weight<T, TM, TWO>(tm, rb, rs, i, unused);
    sm.res_head = h;
    sm.res_tail = tl;
  }
  __syncthreads();
  // Thread 0 locates the segment holding u * W (W accumulated in scan order).
  if (tid == 0) {
    double W = sm.res_head;
    for (int b = 0; b < nblocks; ++b) W += sm.blocks[b];
    W += sm.res_tail;
    const double target = static_cast<double>(u) * W;
    int y = -1;
    int found_block = -1;
    double base = 0.0;
    if (!(W > 0.0)) {
      y = -2;                                        // no mass: degenerate
    } else {
      double C = 0.0;
      for (int i = 0; i < g.head && y < 0; ++i) {
        const double w = scalar_weight<T, TM, TWO>(tm, rb, rs, i, unused);
        if (target < C + w) y = i;
        C += w;
      }
      if (y < 0) {
        for (int b = 0; b < nblocks; ++b) {
          if (target < C + sm.blocks[b]) {
            found_block = b;
            base = C;
            break;
          }
          C += sm.blocks[b];
        }
      }
      if (y < 0 && found_block < 0) {
        int last = -1;
        for (int i = tail0; i < V; ++i) {
          const double w = scalar_weight<T, TM, TWO>(tm, rb, rs, i, unused);
          if (w > 0.0) last = i;
          if (target < C + w) { y = i; break; }
          C += w;
        }
        if (y < 0) y = last;   // rounding at the very end: last positive weight
      }
    }
    sm.res_y = y;
    sm.res_block = found_block;
    sm.res_S = target - base;   // mass still to cover inside the block
  }
  __syncthreads();
  const int blk = sm.res_block;
  if (blk >= 0 && wave == 0) {
    const int v = blk * 64 + lane;
    double l = 0.0;
    double wd[E];
#pragma unroll
    for (int e = 0; e < E; ++e) wd[e] = 0.0;
    if (v < g.nvec) {
      const uint4 vb = load16(rb, g.head, v);
      uint4 vs = make_uint4(0, 0, 0, 0);
      if constexpr (TWO) vs = load16(rs, g.head, v);
      float xb[E], xs[E];
      Elem<T>::unpack(vb, xb);
      Elem<T>::unpack(vs, xs);
      // the same per-element weights (and vector sum) as in the pass above
      if constexpr (A::kPrecise) {
        double w[E];
        tm.weights(xb, xs, w, unused);
#pragma unroll
        for (int e = 0; e < E; ++e) wd[e] = w[e];
      } else {
        float w[E];
        tm.weights(xb, xs, w, unused);
#pragma unroll
        for (int e = 0; e < E; ++e) wd[e] = static_cast<double>(w[e]);
      }
      l = vec_sum<T, TM, TWO>(tm, vb, vs, unused);
    }
    // inclusive scan over lanes
    double incl = l;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double o = __shfl_up(incl, off, 64);
      if (lane >= off) incl += o;
    }
    const double excl = incl - l;
    const double rem = sm.res_S;
    const bool hit = rem < incl && l > 0.0;
    const unsigned long long hits = __ballot(hit);
    int chosen_lane;
    if (hits) {
      chosen_lane = __ffsll(static_cast<long long>(hits)) - 1;
    } else {
      const unsigned long long pos = __ballot(l > 0.0);
      chosen_lane = pos ? 63 - __clzll(static_cast<long long>(pos)) : -1;
    }
    if (lane == chosen_lane) {
      double C = excl;
      int y = -1, last = -1;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if (y < 0) {
          if (wd[e] > 0.0) last = e;
          if (rem < C + wd[e] && wd[e] > 0.0) y = e;
          C += wd[e];
        }
      }
      if (y < 0) y = last;
      sm.res_y = g.head + v * E + y;
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Scalar traversal logic (thread 0)
// ---------------------------------------------------------------------------

struct Params {
  const int32_t* parents;
  const int32_t* tokens;
  const void* target;
  const void* draft;
  const float* uniforms;
  int32_t* accept_len;
  int32_t* accepted_node;
  int32_t* bonus_token;
  int32_t* status;
  int8_t* node_state;
  float* node_theta;
  float* p_init;
  int32_t* counters;
  int num_nodes;
  int vocab;
  int mode;
  float k32;      // log2(e) / T rounded to fp32 (fast element path)
  double k64;     // log2(e) / T (precise element path)
};

// Chain rate of child c given its parent j's current state:
// min(pi_j * b_j(x)/s_j(x), 1) with b/s = [A r - B]_+ * (remaining draft mass).
__device__ inline double child_rate(const TreeSmem& sm, int mode, int j, int c) {
  if (sm.pi[j] == 0.0) return 0.0;
  double v = fmax(sm.A[j] * sm.r0[c] - sm.B[j], 0.0);
  if (mode == TV_SIBLINGS_WITHOUT_REPLACEMENT) v *= sm.rem[j];
  if (v == 0.0) return 0.0;
  return fmin(sm.pi[j] * v, 1.0);
}

// After a pass at j that rejected a child: draft mass left once every rejected
// child's token is removed (Eq. e2 applied to all of them), from the pass's own
// draft-term sum minus those tokens' terms, computed the same way.
__device__ inline void update_remaining_mass(TreeSmem& sm, int j) {
  if (sm.cmd_sd) {
    sm.sdsum[j] = sm.res_sd;
    sm.flags[j] |= kFlagSd;
  }
  const double total = sm.sdsum[j];
  double removed = 0.0;
  const int s0 = sm.child_start[j];
  for (int r = 0; r < sm.next_child[j]; ++r) removed += sm.et[sm.child_list[s0 + r]];
  sm.rem[j] = (total - removed) / total;
}

__device__ inline void issue_stats(TreeSmem& sm, int node, bool two, bool gather) {
  sm.cmd = kCmdStats;
  sm.cmd_node = node;
  sm.cmd_two_rows = two ? 1 : 0;
  sm.cmd_gather = gather ? 1 : 0;
}

__device__ inline void issue_spass(TreeSmem& sm, int node, double alpha, double beta, bool wo) {
  sm.cmd = kCmdSPass;
  sm.cmd_node = node;
  sm.cmd_two_rows = 1;
  sm.cmd_sd = (wo && !(sm.flags[node] & kFlagSd)) ? 1 : 0;
  sm.cmd_ap = alpha * sm.invsb[node];
  sm.cmd_bp = beta * sm.invss[node];
  sm.cmd_cb = sm.cb[node];
  sm.cmd_cs = sm.cs[node];
}

__device__ inline void issue_sample(TreeSmem& sm, int node, bool leaf) {
  sm.cmd = kCmdSample;
  sm.cmd_node = node;
  sm.cmd_cb = sm.cb[node];
  if (leaf) {
    sm.cmd_two_rows = 0;
    sm.cmd_ap = 1.0;
    sm.cmd_bp = 0.0;
    sm.cmd_cs = 0.0;
  } else {
    sm.cmd_two_rows = 1;
    sm.cmd_ap = sm.A[node] * sm.invsb[node];
    sm.cmd_bp = sm.B[node] * sm.invss[node];
    sm.cmd_cs = sm.cs[node];
  }
}

__device__ inline void fail(TreeSmem& sm, int status) {
  sm.status = status;
  sm.cmd = kCmdDone;
}

__device__ inline void init_node_state(TreeSmem& sm, int c, double pi) {
  sm.pi[c] = pi;
  sm.A[c] = 1.0;
  sm.B[c] = 0.0;
  sm.rem[c] = 1.0;
}

// Runs until the next vocabulary pass is needed (or the tree is done).
template <class A>
__device__ __attribute__((noinline)) void advance(TreeSmem& sm, const Params& P, const A& ar) {
  if (sm.cmd == kCmdStats) {
    const int j = sm.cmd_node;
    if (sm.res_bad) { fail(sm, TV_TREE_NONFINITE); return; }
    if (sm.cmd_two_rows) sm.flags[j] |= kFlagStats;
    else sm.flags[j] |= kFlagLeafStats;
  }
  const bool wo = P.mode == TV_SIBLINGS_WITHOUT_REPLACEMENT;
  for (;;) {
    switch (sm.phase) {
      // ---- Alg. 3 initial chain rates for the p_init output -------------
      case kPhPinit: {
        while (sm.pinit_next < P.num_nodes && sm.child_count[sm.pinit_next] == 0)
          ++sm.pinit_next;
        if (sm.pinit_next < P.num_nodes) {
          const int j = sm.pinit_next;
          if (!(sm.flags[j] & kFlagStats)) { issue_stats(sm, j, true, true); return; }
          ++sm.pinit_next;
          continue;
        }
        sm.pini[0] = 1.0;
        for (int i = 1; i < P.num_nodes; ++i) {
          const int j = sm.parent[i];
          if (sm.pini[j] == 0.0) { sm.pini[i] = 0.0; continue; }
          sm.pini[i] = fmin(sm.pini[j] * sm.r0[i], 1.0);
        }
        sm.phase = sm.algo == static_cast<int>(tv::Algo::kTraversal) ? kPhDescend : kPhTlVisit;
        continue;
      }
      // ---- Traversal Verification ----------------------------------------
      case kPhDescend: {   // walk to the first leaf of the remaining tree
        const int j = sm.cur;
        if (sm.next_child[j] < sm.child_count[j]) {
          if (sm.pi[j] > 0.0) {
            if (!(sm.flags[j] & kFlagConsulted)) {
              sm.flags[j] |= kFlagConsulted;
              ++sm.rows_consulted;
            }
            if (!(sm.flags[j] & kFlagStats)) { issue_stats(sm, j, true, true); return; }
          }
          const int c = sm.child_list[sm.child_start[j] + sm.next_child[j]];
          init_node_state(sm, c, child_rate(sm, P.mode, j, c));
          sm.cur = c;
          continue;
        }
        sm.phase = kPhTest;
        continue;
      }
      case kPhTest: {
        const int l = sm.cur;
        if (l == 0) {                       // only the root is left: p(X_0) = 1
          sm.accepted = 0;
          sm.state[0] = TV_NODE_ACCEPTED;
          sm.phase = kPhFinal;
          continue;
        }
        const int j = sm.parent[l];
        if (sm.pi[j] == 0.0) {              // parent can no longer be accepted
          sm.state[l] = TV_NODE_PRUNED;
          sm.theta[l] = 0.0f;
          ++sm.next_child[j];
          sm.cur = j;
          sm.phase = kPhDescend;
          continue;
        }
        const double th = sm.pi[l];
        sm.theta[l] = static_cast<float>(th);
        ++sm.tests;
        if (static_cast<double>(sm.u[l]) < th) {
          sm.state[l] = TV_NODE_ACCEPTED;
          sm.accepted = l;
          sm.phase = kPhFinal;
          continue;
        }
        sm.state[l] = TV_NODE_REJECTED;
        ++sm.next_child[j];
        const double cc = wo ? 1.0 / sm.rem[j] : 1.0;
        sm.alpha = sm.pi[j] * sm.A[j];
        sm.beta = sm.pi[j] * sm.B[j] + cc;
        sm.rejected = l;
        sm.phase = kPhAfterSPass;
        issue_spass(sm, j, sm.alpha, sm.beta, wo);
        return;
      }
      case kPhAfterSPass: {                 // Eq. (e1), (e2), (e3) at the parent
        const int l = sm.rejected;
        const int j = sm.parent[l];
        const double S = sm.res_S;
        ++sm.resid_passes;
        if (S > 0.0) {
          const double inv = 1.0 / S;
          sm.A[j] = sm.alpha * inv;
          sm.B[j] = sm.beta * inv;
          sm.pi[j] = S / (S + (1.0 - sm.pi[j]));
        } else if (j == 0) {
          fail(sm, TV_TREE_DEGENERATE);
          return;
        } else {
          sm.pi[j] = 0.0;
        }
        if (wo) update_remaining_mass(sm, j);
        sm.cur = j;
        sm.phase = kPhDescend;
        continue;
      }
      // ---- Token-level verification --------------------------------------
      case kPhTlVisit: {
        const int j = sm.cur;
        if (sm.child_count[j] == 0) {       // accepted leaf: Y from its target row
          sm.accepted = j;
          if (j == 0) sm.state[0] = TV_NODE_ACCEPTED;
          sm.phase = kPhFinal;
          continue;
        }
        if (!(sm.flags[j] & kFlagConsulted)) {
          sm.flags[j] |= kFlagConsulted;
          ++sm.rows_consulted;
        }
        if (!(sm.flags[j] & kFlagStats)) { issue_stats(sm, j, true, true); return; }
        if (sm.next_child[j] == sm.child_count[j]) {   // all rejected: Y from residual
          sm.accepted = j;
          if (j == 0) sm.state[0] = TV_NODE_ACCEPTED;
          sm.phase = kPhFinal;
          continue;
        }
        const int c = sm.child_list[sm.child_start[j] + sm.next_child[j]];
        const double th = child_rate(sm, P.mode, j, c);
        sm.theta[c] = static_cast<float>(th);
        ++sm.tests;
        if (static_cast<double>(sm.u[c]) < th) {
          sm.state[c] = TV_NODE_ACCEPTED;
          init_node_state(sm, c, 1.0);
          sm.cur = c;
          continue;
        }
        sm.state[c] = TV_NODE_REJECTED;
        ++sm.next_child[j];
        const double cc = wo ? 1.0 / sm.rem[j] : 1.0;
        sm.alpha = sm.A[j];
        sm.beta = sm.B[j] + cc;
        sm.rejected = c;
        sm.phase = kPhTlAfterSPass;
        issue_spass(sm, j, sm.alpha, sm.beta, wo);
        return;
      }
      case kPhTlAfterSPass: {               // Algorithm 2 rejection branch
        const int c = sm.rejected;
        const int j = sm.parent[c];
        const double S = sm.res_S;
        ++sm.resid_passes;
        if (!(S > 0.0)) { fail(sm, TV_TREE_DEGENERATE); return; }
        const double inv = 1.0 / S;
        sm.A[j] = sm.alpha * inv;
        sm.B[j] = sm.beta * inv;
        if (wo) update_remaining_mass(sm, j);
        sm.phase = kPhTlVisit;
        continue;
      }
      // ---- Final sample Y --------------------------------------------------
      case kPhFinal: {
        const int a = sm.accepted;
        if (sm.child_count[a] == 0) {
          sm.phase = kPhFinalLeafStats;
          if (!(sm.flags[a] & kFlagLeafStats)) { issue_stats(sm, a, false, false); return; }
          continue;
        }
        sm.phase = kPhAfterSample;
        issue_sample(sm, a, false);
        return;
      }
      case kPhFinalLeafStats: {
        sm.phase = kPhAfterSample;
        issue_sample(sm, sm.accepted, true);
        return;
      }
      case kPhAfterSample: {
        if (sm.res_y < 0) { fail(sm, TV_TREE_DEGENERATE); return; }
        sm.cmd = kCmdDone;
        return;
      }
      default:
        fail(sm, TV_TREE_DEGENERATE);
        return;
    }
  }
}

// ---------------------------------------------------------------------------
// The kernel: one workgroup per tree
// ---------------------------------------------------------------------------

template <typename T, class A, int algo>
__global__ void __launch_bounds__(kThreads) verify_kernel(Params P, A ar) {
  __shared__ TreeSmem sm;
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const int n1 = P.num_nodes;
  const int V = P.vocab;
  const size_t tree_off = static_cast<size_t>(b) * n1;
  const T* zb = static_cast<const T*>(P.target) + tree_off * V;
  const T* zs = static_cast<const T*>(P.draft) + tree_off * V;

  // ---- load and check the tree -----------------------------------------
  if (tid == 0) {
    sm.status = TV_TREE_OK;
    sm.res_bad = 0;
  }
  __syncthreads();
  int bad_parent = 0, bad_token = 0;
  for (int i = tid; i < n1; i += kThreads) {
    const int p = P.parents[tree_off + i];
    const int x = P.tokens[tree_off + i];
    if (i == 0 ? p != -1 : (p < 0 || p >= i)) bad_parent = 1;
    if (i > 0 && (x < 0 || x >= V)) bad_token = 1;
    sm.parent[i] = static_cast<int16_t>(i == 0 ? -1 : (p < 0 || p >= i ? 0 : p));
    sm.token[i] = x;
    sm.u[i] = P.uniforms[tree_off + i];
    sm.child_count[i] = 0;
    sm.next_child[i] = 0;
    sm.state[i] = TV_NODE_UNTESTED;
    sm.flags[i] = 0;
    sm.theta[i] = -1.0f;
    sm.pini[i] = -1.0;
  }
  bad_parent = __syncthreads_or(bad_parent);
  bad_token = __syncthreads_or(bad_token);
  if (tid == 0) {
    if (bad_parent) sm.status = TV_TREE_BAD_PARENT;
    else if (bad_token) sm.status = TV_TREE_BAD_TOKEN;
  }
  __syncthreads();
  if (sm.status == TV_TREE_OK) {
    for (int i = 1 + tid; i < n1; i += kThreads) atomicAdd(&sm.child_count[sm.parent[i]], 1);
    __syncthreads();
    if (tid == 0) {
      int start = 0;
      for (int j = 0; j < n1; ++j) {
        sm.child_start[j] = static_cast<int16_t>(start);
        start += sm.child_count[j];
      }
    }
    __syncthreads();
    // rank among siblings = earlier nodes with the same parent
    for (int i = 1 + tid; i < n1; i += kThreads) {
      const int p = sm.parent[i];
      int rank = 0, d = 1;
      for (int k2 = 1; k2 < i; ++k2) rank += (sm.parent[k2] == p);
      for (int a = p; a > 0; a = sm.parent[a]) ++d;
      sm.child_list[sm.child_start[p] + rank] = static_cast<int16_t>(i);
      sm.depth[i] = static_cast<int16_t>(d);
    }
    if (tid == 0) sm.depth[0] = 0;
    __syncthreads();
    int dup = 0;
    if (P.mode == TV_SIBLINGS_WITHOUT_REPLACEMENT) {
      for (int i = 1 + tid; i < n1; i += kThreads) {
        const int p = sm.parent[i];
        const int s0 = sm.child_start[p], cnt = sm.child_count[p];
        for (int r = 0; r < cnt; ++r) {
          const int c = sm.child_list[s0 + r];
          if (c > i && sm.token[c] == sm.token[i]) dup = 1;
        }
      }
    }
    dup = __syncthreads_or(dup);
    if (tid == 0 && dup) sm.status = TV_TREE_DUP_SIBLING;
    __syncthreads();
  }

  // ---- traversal ---------------------------------------------------------
  if (sm.status == TV_TREE_OK) {
    if (tid == 0) {
      sm.algo = algo;
      sm.cur = 0;
      sm.accepted = -1;
      sm.rows_consulted = sm.resid_passes = sm.tests = 0;
      sm.pinit_next = 0;
      init_node_state(sm, 0, 1.0);
      sm.res_y = -1;
      sm.cmd = -1;
      sm.cmd_sd = 0;
      if (P.p_init && algo == static_cast<int>(tv::Algo::kTraversal)) sm.phase = kPhPinit;
      else if (algo == static_cast<int>(tv::Algo::kTraversal)) sm.phase = kPhDescend;
      else sm.phase = kPhTlVisit;
      advance(sm, P, ar);
    }
    __syncthreads();
    for (;;) {
      const int cmd = sm.cmd;
      if (cmd == kCmdDone) break;
      const int node = sm.cmd_node;
      const T* rb = zb + static_cast<size_t>(node) * V;
      const T* rs = zs + static_cast<size_t>(node) * V;
      if (cmd == kCmdStats) {
        if (sm.cmd_two_rows) stats_pass<T, A, true>(sm, rb, rs, V, ar, node, sm.cmd_gather != 0);
        else stats_pass<T, A, false>(sm, rb, rs, V, ar, node, false);
      } else {
        const TermParams tp{sm.cmd_cb, sm.cmd_cs, sm.cmd_ap, sm.cmd_bp};
        if (cmd == kCmdSPass) {
          if (sm.cmd_sd) s_pass<T, A, true>(sm, rb, rs, V, ar, tp);
          else s_pass<T, A, false>(sm, rb, rs, V, ar, tp);
        } else if (sm.cmd_two_rows) {
          sample_pass<T, A, true>(sm, rb, rs, V, ar, tp, sm.u[0]);
        } else {
          sample_pass<T, A, false>(sm, rb, rs, V, ar, tp, sm.u[0]);
        }
      }
      if (tid == 0) advance(sm, P, ar);
      __syncthreads();
    }
  }

  // ---- outputs -------------------------------------------------------------
  const bool ok = sm.status == TV_TREE_OK;
  for (int i = tid; i < n1; i += kThreads) {
    if (P.node_state) P.node_state[tree_off + i] = ok ? static_cast<int8_t>(sm.state[i]) : 0;
    if (P.node_theta) P.node_theta[tree_off + i] = ok ? sm.theta[i] : -1.0f;
    if (P.p_init) P.p_init[tree_off + i] = ok ? static_cast<float>(sm.pini[i]) : -1.0f;
  }
  if (tid == 0) {
    P.status[b] = sm.status;
    P.accept_len[b] = ok ? sm.depth[sm.accepted] : -1;
    P.accepted_node[b] = ok ? sm.accepted : -1;
    P.bonus_token[b] = ok ? sm.res_y : -1;
    if (P.counters) {
      int32_t* c = P.counters + static_cast<size_t>(b) * TV_NUM_COUNTERS;
      c[0] = ok ? sm.rows_consulted : 0;
      c[1] = ok ? sm.resid_passes : 0;
      c[2] = ok ? (sm.child_count[sm.accepted] == 0 ? 1 : 0) : 0;
      c[3] = ok ? sm.tests : 0;
    }
  }
}

// Vocabularies below this use the precise element path whatever the dtype:
// with few elements the per-element rounding of the fast path does not average.
constexpr int kPreciseBelowVocab = 16384;

template <typename T, int algo>
int launch_typed(const Params& P, bool precise, int batch, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(batch));
  const dim3 block(kThreads);
  if (precise) {
    PreciseArith ar{P.k64};
    hipLaunchKernelGGL((verify_kernel<T, PreciseArith, algo>), grid, block, 0, stream, P, ar);
  } else {
    FastArith ar{P.k32};
    hipLaunchKernelGGL((verify_kernel<T, FastArith, algo>), grid, block, 0, stream, P, ar);
  }
  return hipGetLastError() == hipSuccess ? TV_OK : TV_ERR_HIP;
}

}  // namespace

namespace tv {

int launch(const VerifyArgs& a, Algo algo, hipStream_t stream) {
  Params P;
  P.parents = a.parents;
  P.tokens = a.tokens;
  P.target = a.target;
  P.draft = a.draft;
  P.uniforms = a.uniforms;
  P.accept_len = a.accept_len;
  P.accepted_node = a.accepted_node;
  P.bonus_token = a.bonus_token;
  P.status = a.status;
  P.node_state = a.node_state;
  P.node_theta = a.node_theta;
  P.p_init = a.p_init;
  P.counters = a.counters;
  P.num_nodes = a.num_nodes;
  P.vocab = a.vocab;
  P.mode = a.mode;
  P.k64 = 1.4426950408889634 / static_cast<double>(a.temperature);
  P.k32 = static_cast<float>(P.k64);
  const bool precise = a.dtype == TV_DTYPE_F32 || a.vocab < kPreciseBelowVocab;
  constexpr int kTv = static_cast<int>(Algo::kTraversal);
  constexpr int kTl = static_cast<int>(Algo::kTokenLevel);
  if (a.dtype == TV_DTYPE_BF16)
    return algo == Algo::kTraversal ? launch_typed<uint16_t, kTv>(P, precise, a.batch, stream)
                                    : launch_typed<uint16_t, kTl>(P, precise, a.batch, stream);
  return algo == Algo::kTraversal ? launch_typed<float, kTv>(P, precise, a.batch, stream)
                                  : launch_typed<float, kTl>(P, precise, a.batch, stream);
}

}  // namespace tv
