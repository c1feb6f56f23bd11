// Traversal Verification (arXiv 2505.12398, Algorithm 3) and the token-level
// baseline (Sec. 2.2, Algorithm 2 per node) for gfx950 (MI355X, CDNA4).
//
// Work split. Each tree is verified by a group of G workgroups (G chosen per
// launch so that the groups fill the device: G is large for small batches and
// small for large ones). Every member of a group holds the tree in LDS and runs
// the same sequential traversal on its thread 0, on the same data, so all
// members take the same decisions. Whenever the traversal needs vocabulary-wide
// quantities, each member computes its fixed 1/G stripe of the rows involved,
// publishes the stripe's partial results and waits for the other members';
// every member then combines the G partials in member order and continues.
// The group only exchanges these partials, a few words per member and pass.
// The launch is cooperative, so all members of a group are resident together.
// A group with no tree left lends its workgroups to running groups as
// helpers: a helper takes stripes of another group's passes (the group's
// member 0 publishes each batch for them), so the trees that run longest get
// more workgroups as the others finish. With helpers the number of stripes
// of a pass depends on timing, and so do the last bits of the sums.
//
// Pass kinds:
//   STATS   per row: maximum and sum of 2^(z*k - max*k), k = log2(e)/T, over
//           the target and draft rows of a node (the target row only for an
//           accepted leaf); issued the first time the traversal descends into
//           a node whose acceptance rate is above zero;
//   SPASS   S = sum_x [alpha p(x) - beta q(x)]_+ over the parent's rows, one per
//           rejection: Eq. (e1) and (e3);
//   WSUM    the same weights as SPASS without updating anything (only needed
//           when Y is drawn at a node whose last pass was not its SPASS).
// Passes are issued in batches: the pass the traversal needs now plus the
// STATS passes of the internal nodes it will descend into next (the nodes on
// the leftmost remaining path below the next child); those depend only on
// their own rows, so they are computed with it instead of one after another.
// Y is drawn by inverse CDF in ascending token order: the stripe partials of
// the pass that produced the weights locate the stripe holding u*W, and one
// member rescans that stripe.
//
// A node's residual target and draft are never materialised: after k
// rejections they are b = [A p - B q]_+ and s = c q off the rejected tokens,
// so four scalars (pi, A, B, remaining draft mass) carry Eq. (e1)-(e3) and a
// sibling's ratio b/s = [A r - B]_+ / c needs no vocabulary pass.
//
// Precision. Logits are widened exactly to fp32 and every per-node scalar is
// fp64. FAST (bf16 logits with V >= 16384) takes each term as the hardware
// exp2 of an fp32 fma and accumulates in fp64; PRECISE (fp32 logits, or any
// V < 16384) evaluates every term in fp64. The remaining draft mass after Eq.
// (e2) is the pass's own sum of draft terms minus the rejected tokens' terms,
// never 1 - sum q(rejected), which cancels when those held most of the mass.
// Every sum is formed in a fixed order (per thread, across the workgroup, then
// across members), so results are reproducible for a given group size.
//
// Synchronisation. A member writes each partial as four 64-bit words with
// agent-scope atomic stores; every word carries the batch's 16-bit tag (in the
// lowest mantissa bits of a sum, in the zero low bits of a float maximum
// widened to double). Members poll the G partials of a pass with agent-scope
// atomic loads until all words carry the expected tag: 64-bit accesses are
// single-copy atomic, so each word read is whole, and no counter, fence or
// second round of loads is needed; agent-scope atomic loads see other
// workgroups' atomic stores without a cache invalidation. Partials are double
// buffered by batch parity, so batch k+1 never overwrites what a member may
// still be reading of batch k, and every entry is rewritten at least every 14
// batches, so an entry left from an earlier batch never carries the tag being
// awaited. Every wait is bounded by a wall-clock limit after which the launch
// is abandoned (trees not finished then report TV_TREE_ABORTED), so no wave
// can spin forever.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include <mutex>
#include <type_traits>

#include "tv.h"
#include "tv_launch.h"

namespace {

constexpr int kNT = 256;                       // threads per workgroup
constexpr int kNW = kNT / 64;
// vectors per row in flight per lane: the fp64 element path needs more registers
template <class A> constexpr int kUnrollOf = A::kPrecise ? 2 : 4;
constexpr int kCapSmall = 128;                 // node capacity of the compact variant
constexpr int kCapLarge = TV_MAX_NODES;
constexpr int kMaxBatch = tv::kMaxBatchPasses; // passes per batch
constexpr int kMaxGroup = tv::kMaxGroup;       // workgroups per tree
static_assert(kMaxGroup <= 64, "member partials are combined by one wavefront");

// Pass kinds and controller commands.
enum : int {
  kCmdNone = 0, kCmdStats2 = 1, kCmdStats1 = 2, kCmdSPass = 3, kCmdSPassSd = 4, kCmdWSum = 5,
  kCmdLocalSample = 6, kCmdDone = 7, kCmdBatch = 8, kCmdAbandon = 9
};
enum : int {
  kPhDescend = 0, kPhTest, kPhAfterSPass, kPhFinal, kPhFinalLeafStats, kPhFinalWSum,
  kPhAfterSample, kPhPinit, kPhTlVisit, kPhTlAfterSPass
};
enum : uint8_t {
  kFlagStats = 1, kFlagConsulted = 2, kFlagBad = 4, kFlagSd = 8,
  kFlagPrunedBelow = 16     // children from prune_from on, and their subtrees, are pruned
};

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
  const float* tmax;         // row statistics given by the caller, or NULL (see tv_verify_stats)
  const double* tsum;
  const float* dmax;
  const double* dsum;
  uint8_t* ws;
  size_t off_parts, parts_words;
  size_t off_desc, desc_words;
  long long spin_limit;      // wall-clock ticks a wait may last before the launch is abandoned
  int batch;
  int num_nodes;
  int vocab;
  int mode;
  int algo;
  int early;                 // skip updates that decide nothing (node_theta not asked for)
  int G;                     // workgroups per group (per tree)
  int Gx;                    // most contributors (members + helpers) a group's pass has
  int ngroups;               // groups; group g verifies trees g, g + ngroups, ...
  float k32;                 // log2(e) / T rounded to fp32 (fast element path)
  double k64;                // log2(e) / T (precise element path)
};

// A reference into LDS with its address space in the type, so that functions
// the compiler does not inline still access it with LDS instructions rather
// than through generic pointers.
template <class X> using Lds = __attribute__((address_space(3))) X;
template <class X>
__device__ __forceinline__ Lds<X>& lds_ref(X& x) {
  return *reinterpret_cast<Lds<X>*>((__attribute__((address_space(3))) void*)&x);
}

// One contributor's partial result of one pass: four 64-bit words (two sums,
// two maxima), each written and read with a single-copy atomic 64-bit access
// and each carrying the batch's 16-bit tag, so a reader that sees the tag in
// all four words has the whole result of that batch. The sums are >= 0 (or
// NaN): the tag replaces their 16 lowest mantissa bits (a relative change
// below 2^-36). The maxima are floats widened to doubles, whose low 29
// mantissa bits are 0: bits 0-15 hold the tag, bits 16-21 a small count
// (member 0 reports the number of helpers for the next batch in the draft
// maximum of pass 0).
struct SegPart {
  uint64_t w[4];
};

// Tag of batch `seq` (1, 2, ...): never 0, the value of a cleared entry
// (entries are cleared before each launch).
__device__ __forceinline__ uint64_t batch_tag(uint32_t seq) {
  return 0x8000u | (seq & 0x7FFFu);
}

constexpr uint64_t kTagMask = 0xFFFFull;
constexpr uint64_t kMaxMeta = 0x3FFFFFull;     // tag and count bits of a maximum
__device__ __forceinline__ uint64_t enc_sum(double v, uint64_t tag) {
  return (static_cast<uint64_t>(__double_as_longlong(v)) & ~kTagMask) | tag;
}
__device__ __forceinline__ double dec_sum(uint64_t w) {
  return __longlong_as_double(static_cast<long long>(w & ~kTagMask));
}
__device__ __forceinline__ uint64_t enc_max(float v, uint64_t tag, uint64_t count = 0) {
  return static_cast<uint64_t>(__double_as_longlong(static_cast<double>(v))) | tag |
         (count << 16);
}
__device__ __forceinline__ float dec_max(uint64_t w) {
  return static_cast<float>(__longlong_as_double(static_cast<long long>(w & ~kMaxMeta)));
}
__device__ __forceinline__ int max_count(uint64_t w) { return static_cast<int>((w >> 16) & 63u); }
__device__ __forceinline__ bool tags_are(const uint64_t (&w)[4], uint64_t tag) {
  return (w[0] & kTagMask) == tag && (w[1] & kTagMask) == tag && (w[2] & kTagMask) == tag &&
         (w[3] & kTagMask) == tag;
}

// The sums and maxima a stripe pass produces.
struct StripeResult {
  double s0, s1;
  float m0, m1;
};

// ---------------------------------------------------------------------------
// Workspace access and synchronisation primitives
// ---------------------------------------------------------------------------

template <class PP>
__device__ __forceinline__ uint32_t* ws_abort(const PP& P) {
  return reinterpret_cast<uint32_t*>(P.ws);
}
// partial of member m for pass p of the batch with parity `par` in group g
template <class PP>
__device__ __forceinline__ SegPart* ws_parts(const PP& P, int g, int par, int p) {
  return reinterpret_cast<SegPart*>(P.ws + P.off_parts) +
         ((static_cast<size_t>(g) * 2 + par) * kMaxBatch + p) * P.Gx;
}

__device__ __forceinline__ uint64_t ld_rlx(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_rlx(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_rlx(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_rlx(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

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
  // a value of the row (or an infinity) back into its own format, exactly
  __device__ static inline uint16_t narrow(float x) {
    return static_cast<uint16_t>(__float_as_uint(x) >> 16);
  }
  __device__ static inline float widen(uint16_t v) {
    return __uint_as_float(static_cast<uint32_t>(v) << 16);
  }
};

template <> struct Elem<float> {
  static constexpr int E = 4;
  __device__ static inline void unpack(const uint4& v, float (&x)[4]) {
    x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y);
    x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
  }
  __device__ static inline float scalar(const float* p) { return *p; }
  __device__ static inline float narrow(float x) { return x; }
  __device__ static inline float widen(float v) { return v; }
};

// A row split into a scalar head (up to the first 16-byte boundary), full
// 16-byte vectors, and a scalar tail. Target and draft rows of a node share
// the same split (the host checks the two tensors agree modulo 16 bytes).
struct Geom {
  int head, nvec, tail;
};

template <typename T>
__device__ __forceinline__ Geom row_geom(const T* row, int V) {
  constexpr int E = Elem<T>::E;
  const int mis = static_cast<int>(reinterpret_cast<uintptr_t>(row) & 15);
  int head = mis ? (16 - mis) / static_cast<int>(sizeof(T)) : 0;
  head = head < V ? head : V;
  const int rest = V - head;
  return Geom{head, rest / E, rest % E};
}

// The stripe of member m of G: vectors [vb, ve); member 0 also holds the head
// elements and member G-1 the tail elements.
struct SegRange {
  int vb, ve;
  bool first, last;
};

__device__ __forceinline__ SegRange stripe(const Geom& g, int m, int G) {
  SegRange r;
  r.vb = static_cast<int>((static_cast<long long>(g.nvec) * m) / G);
  r.ve = static_cast<int>((static_cast<long long>(g.nvec) * (m + 1)) / G);
  r.first = m == 0;
  r.last = m == G - 1;
  return r;
}

template <typename T>
__device__ __forceinline__ uint4 load16(const T* row, int head, int v) {
  return *reinterpret_cast<const uint4*>(row + head + v * Elem<T>::E);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Keeps a loaded vector where it is: without this the compiler may sink a load
// into the guarded arithmetic that uses it and serialise a round's loads.
__device__ __forceinline__ void pin(uint4& v) {
  asm volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
}

// ---------------------------------------------------------------------------
// Workgroup reductions (fixed order: deterministic). Results valid in every thread.
// ---------------------------------------------------------------------------

struct WgScratch {
  double red_d[2 * kNW];
  float red_f[2 * kNW];
  double scan_d[kNW];
  int stop;                 // the launch was abandoned
  int hit;                  // first thread whose range holds the sample
  int last_pos;             // last thread with positive weight
  int smp_seg;
  int smp_chunk;            // chunk of the stripe holding the sample (-1: none yet)
  int smp_last_chunk;       // last chunk with positive mass
  double smp_target;        // mass still to cover inside the chosen stripe / chunk
  double smp_window;        // mass of the window of chunks just scanned
  double smp_chunks[256];   // chunk sums of one window
  int hnext;                // helpers member 0 reported for the next batch
  StripeResult res[kMaxBatch];   // this workgroup's results of the batch's passes
  uint64_t res_count;            // the count member 0 reports with them
  // a helper's view of the group it helps
  int help_g, help_h, help_state;
  uint32_t d_seq;
  int d_tree, d_bn, d_geff;
  int16_t d_node[8];
  int8_t d_cmd[8];
  double d_ap, d_bp, d_cb, d_cs;
};

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

template <class WS>
__device__ __forceinline__ void block_sum2(WS& ws, double& a, double& b) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  a = wave_sum(a);
  b = wave_sum(b);
  if (lane == 0) {
    ws.red_d[wave] = a;
    ws.red_d[kNW + wave] = b;
  }
  __syncthreads();
  double ta = 0.0, tb = 0.0;
#pragma unroll
  for (int w = 0; w < kNW; ++w) {
    ta += ws.red_d[w];
    tb += ws.red_d[kNW + w];
  }
  __syncthreads();
  a = ta;
  b = tb;
}

template <class WS>
__device__ __forceinline__ void block_max2(WS& ws, float& a, float& b) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  a = wave_max(a);
  b = wave_max(b);
  if (lane == 0) {
    ws.red_f[wave] = a;
    ws.red_f[kNW + wave] = b;
  }
  __syncthreads();
  float ta = -INFINITY, tb = -INFINITY;
#pragma unroll
  for (int w = 0; w < kNW; ++w) {
    ta = fmaxf(ta, ws.red_f[w]);
    tb = fmaxf(tb, ws.red_f[kNW + w]);
  }
  __syncthreads();
  a = ta;
  b = tb;
}

// Inclusive scan over the threads of the workgroup in thread order.
template <class WS>
__device__ __forceinline__ double block_incl_scan(WS& ws, double v) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  double incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  if (lane == 63) ws.scan_d[wave] = incl;
  __syncthreads();
  double base = 0.0;
  for (int w = 0; w < wave; ++w) base += ws.scan_d[w];
  __syncthreads();
  return base + incl;
}

// ---------------------------------------------------------------------------
// Element arithmetic. A row's terms are 2^(z*k + c) for a frame offset c
// (c = -max * k once the row maximum is known).
// ---------------------------------------------------------------------------

struct FastArith {                 // hardware exp2 of an fp32 fma
  static constexpr bool kPrecise = false;
  float k;                         // log2(e) / T rounded to fp32
  __device__ double frame(float m) const { return static_cast<double>(-m * k); }
  // 2^(frame(m) + m k): the rounding of the fp32 product in frame(m). A row
  // sum given in the exact frame of its maximum times this is the sum of the
  // terms 2^(z k + frame(m)) this arithmetic forms.
  __device__ double frame_rounding(float m) const {
    return exp2(frame(m) + static_cast<double>(m) * static_cast<double>(k));
  }
  __device__ double ex(float z, double c) const {
    return static_cast<double>(fast_exp2(fmaf(z, k, static_cast<float>(c))));
  }
  __device__ double kd() const { return static_cast<double>(k); }
};

struct PreciseArith {              // fp64 throughout
  static constexpr bool kPrecise = true;
  double k;                        // log2(e) / T
  __device__ double frame(float m) const { return -static_cast<double>(m) * k; }
  __device__ double frame_rounding(float) const { return 1.0; }
  __device__ double ex(float z, double c) const {
    return exp2(fma(static_cast<double>(z), k, c));
  }
  __device__ double kd() const { return k; }
};

// Running maximum and sum of one thread over a row. Before the first finite
// value the maximum is -inf and the frame is that of a finite sentinel, so
// -inf entries add 2^-inf = 0 with no branch, a NaN or +inf entry turns the
// sum into NaN, and a row with no finite entry keeps maximum -inf.
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
__device__ __forceinline__ void online_add(Online& o, const float (&x)[N], const A& ar) {
  float vmax = x[0];
#pragma unroll
  for (int e = 1; e < N; ++e) vmax = fmaxf(vmax, x[e]);
  online_raise(o, vmax, ar);
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

// Residual weights max(ap * tb - bp * ts, 0), tb and ts the target and draft
// terms of an element (TWO == false: target only, weight ap * tb). With SD the
// draft terms are also summed, exactly in fp64.
struct TermParams {
  double cb, cs;   // frames of the target and draft rows
  double ap, bp;   // multipliers of the target and draft terms
};

template <class A, bool TWO, bool SD> struct Terms;

template <bool TWO, bool SD> struct Terms<FastArith, TWO, SD> {
  using W = float;
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

template <bool TWO, bool SD> struct Terms<PreciseArith, TWO, SD> {
  using W = double;
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

// One unit of a segment: a scalar element or a 16-byte vector.
template <typename T, class TM, bool TWO>
__device__ __forceinline__ double vec_sum(const TM& tm, const uint4& vb, const uint4& vs,
                                          double& sd) {
  constexpr int E = Elem<T>::E;
  float xb[E], xs[E];
  Elem<T>::unpack(vb, xb);
  if constexpr (TWO) {
    Elem<T>::unpack(vs, xs);
  } else {
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

// One round of loads: vectors v0 + u * kNT (u < U) of both rows, clamped to
// vmax so that every load is issued unconditionally.
template <typename T, bool TWO, int U>
struct Round {
  uint4 b[U], s[U];
  __device__ __forceinline__ void load(const T* rb, const T* rs, int head, int v0, int vmax) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = min(v0 + u * kNT, vmax);
      b[u] = load16(rb, head, v);
      if constexpr (TWO) s[u] = load16(rs, head, v);
    }
  }
  __device__ __forceinline__ void pin_all() {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      pin(b[u]);
      if constexpr (TWO) pin(s[u]);
    }
  }
};

// Calls f(target vector, draft vector) for every vector of the stripe this
// thread owns (vb + tid + i * kNT), in that order. Each step issues two rounds
// of loads before any arithmetic and consumes the first round while the
// second is still in flight. Loads past the stripe are clamped re-reads of its
// last vector. With kShort, a step whose stripe ends within its first round
// issues no second round (whose loads would otherwise still be waited for):
// the large-tree variant, whose stripes are short; the compact variant keeps
// the loop as it is, where the branch measured slower.
template <typename T, bool TWO, int U, bool kShort = false, class F>
__device__ __forceinline__ void stream_stripe(const T* rb, const T* rs, int head,
                                              const SegRange& r, F&& f) {
  constexpr int kRound = kNT * U;
  const int tid = threadIdx.x;
  const int vmax = r.ve - 1;
  auto consume = [&](Round<T, TWO, U>& q, int base) {
    q.pin_all();
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (base + tid + u * kNT < r.ve) f(q.b[u], q.s[u]);
  };
#pragma unroll 1
  for (int base = r.vb; base < r.ve; base += 2 * kRound) {
    Round<T, TWO, U> x, y;
    const bool second = !kShort || base + kRound < r.ve;
    x.load(rb, rs, head, base + tid, vmax);
    if (second) y.load(rb, rs, head, base + kRound + tid, vmax);
    __builtin_amdgcn_sched_barrier(0);
    consume(x, base);
    if (second) consume(y, base + kRound);
  }
}

// ---------------------------------------------------------------------------
// Stripe passes. Thread t takes vectors vb + t + i * kNT of the stripe; per
// thread: head elements, vectors in order, tail elements. Loads are
// unconditional (indices clamped into the stripe) so that all of a round's
// loads are in flight together; only the arithmetic is guarded.
// ---------------------------------------------------------------------------

template <typename T, class A, bool TWO, bool kShort>
__device__ void stripe_stats(Lds<WgScratch>& ws, const T* rb, const T* rs, const Geom& g,
                             const SegRange& r, const A& ar, StripeResult& out) {
  constexpr int E = Elem<T>::E;
  const int tid = threadIdx.x;
  Online ob = online_init(ar), os = online_init(ar);
  if (r.first && tid < g.head) {
    float xb[1] = {Elem<T>::scalar(rb + tid)};
    online_add(ob, xb, ar);
    if constexpr (TWO) {
      float xs[1] = {Elem<T>::scalar(rs + tid)};
      online_add(os, xs, ar);
    }
  }
  stream_stripe<T, TWO, kUnrollOf<A>, kShort>(rb, rs, g.head, r, [&](const uint4& vb, const uint4& vs) {
    float x[E];
    Elem<T>::unpack(vb, x);
    online_add(ob, x, ar);
    if constexpr (TWO) {
      Elem<T>::unpack(vs, x);
      online_add(os, x, ar);
    }
  });
  if (r.last && tid < g.tail) {
    const int i = g.head + g.nvec * E + tid;
    float xb[1] = {Elem<T>::scalar(rb + i)};
    online_add(ob, xb, ar);
    if constexpr (TWO) {
      float xs[1] = {Elem<T>::scalar(rs + i)};
      online_add(os, xs, ar);
    }
  }
  float Mb = ob.m, Ms = TWO ? os.m : -INFINITY;
  block_max2(ws, Mb, Ms);
  // exact fp64 change of frame; a thread that saw no finite value has s = 0
  // (or NaN) and the factor 0. A stripe with no finite value keeps s = 0 (or
  // NaN) and maximum -inf.
  double Sb = (Mb > -INFINITY) ? ob.s * exp2(ar.frame(Mb) - ob.c) : ob.s;
  double Ss = (TWO && Ms > -INFINITY) ? os.s * exp2(ar.frame(Ms) - os.c) : (TWO ? os.s : 0.0);
  block_sum2(ws, Sb, Ss);
  out.m0 = Mb;
  out.m1 = Ms;
  out.s0 = Sb;
  out.s1 = Ss;
}

template <typename T, class A, bool SD, bool kShort>
__device__ void stripe_wsum(Lds<WgScratch>& ws, const T* rb, const T* rs, const Geom& g,
                            const SegRange& r, const A& ar, const TermParams& p,
                            StripeResult& out) {
  const Terms<A, true, SD> tm(ar, p);
  using TM = Terms<A, true, SD>;
  const int tid = threadIdx.x;
  double acc = 0.0, sd = 0.0;
  if (r.first && tid < g.head) acc += scalar_weight<T, TM, true>(tm, rb, rs, tid, sd);
  stream_stripe<T, true, kUnrollOf<A>, kShort>(rb, rs, g.head, r, [&](const uint4& vb, const uint4& vs) {
    acc += vec_sum<T, TM, true>(tm, vb, vs, sd);
  });
  if (r.last && tid < g.tail)
    acc += scalar_weight<T, TM, true>(tm, rb, rs, g.head + g.nvec * Elem<T>::E + tid, sd);
  block_sum2(ws, acc, sd);
  out.s0 = acc;
  out.s1 = sd;
  out.m0 = 0.0f;
  out.m1 = 0.0f;
}

// ---------------------------------------------------------------------------
// Tree state (LDS) and the scalar traversal logic (thread 0)
// ---------------------------------------------------------------------------

template <int kCap>
struct TreeSmem {
  // tree structure
  int16_t parent[kCap];
  int16_t child_start[kCap];
  int16_t child_list[kCap];
  int16_t next_child[kCap];        // children already removed (always a prefix)
  int16_t rank[kCap];              // position among the parent's children
  int16_t prune_from[kCap];        // with kFlagPrunedBelow: first pruned child
  int32_t child_count[kCap];
  int32_t token[kCap];
  float u[kCap];
  float theta[kCap];
  float gb[kCap], gs[kCap];        // parent's target / draft logit at the node's token
                                   // (gathered when the tree is loaded)
  uint8_t state[kCap];
  uint8_t flags[kCap];
  // per-node verification state
  double pi[kCap];                 // current acceptance rate p of the chain ending here
  double A[kCap];                  // residual target b = [A p - B q]_+
  double B[kCap];
  double rem[kCap];                // draft mass left after removing rejected tokens
  double removed[kCap];            // draft terms of the rejected children's tokens
  double pini[kCap];
  double sdsum[kCap];              // sum of the draft row's terms in its frame
  double invsb[kCap];              // 1 / (sum of the target row's terms)
  double invss[kCap];              // 1 / (sum of the draft row's terms)
  double cb[kCap];                 // exponent offset of the target row: -max * k
  double cs[kCap];                 // exponent offset of the draft row
  double r0[kCap];                 // original ratio p(x) / q(x) of the node's token at its parent
  double et[kCap];                 // draft term of the node's token in the parent's frame
  // traversal state (held in registers while the controller runs)
  int has_tree, tree;
  int phase, cur, accepted, rejected, status;
  int rows_consulted, resid_passes, tests, pinit_next;
  int any_pruned;                  // some node has kFlagPrunedBelow
  double alpha, beta;
  // command from the controller; a batch: pass 0 is the one the traversal
  // waits for, the others are STATS of nodes it will descend into
  int cmd;
  int bn;
  int16_t bnode[kMaxBatch];
  int8_t bcmd[kMaxBatch];
  double cmd_ap, cmd_bp, cmd_cb, cmd_cs;    // parameters of a SPASS / WSUM pass 0
  // the batch in flight, then just completed
  int pending;
  uint32_t seq;                    // batches this group has run (all trees so far)
  int geff;                        // contributors (members + helpers) of the next batch
  int geff_last;                   // contributors of the batch just completed
  int spass_node;                  // node whose SPASS partials are in the workspace (-1: none)
  double last_ap, last_bp, last_cb, last_cs;
  // local sample request
  int smp_from_stats;              // segment weights from a STATS pass (accepted leaf)
  int smp_two;
  double smp_ap, smp_bp, smp_cb, smp_cs;
  // results of the combine
  double res_S, res_sd;
  int res_y;
};

// Chain rate of child c given its parent j's current state:
// min(pi_j * b_j(x)/s_j(x), 1) with b/s = [A r - B]_+ * (remaining draft mass).
template <int kCap>
__device__ inline double child_rate(const Lds<TreeSmem<kCap>>& sm, int mode, int j, int c) {
  if (sm.pi[j] == 0.0) return 0.0;
  double v = fmax(sm.A[j] * sm.r0[c] - sm.B[j], 0.0);
  if (mode == TV_SIBLINGS_WITHOUT_REPLACEMENT) v *= sm.rem[j];
  if (v == 0.0) return 0.0;
  return fmin(sm.pi[j] * v, 1.0);
}

// After a pass at j that rejected child l: draft mass left once every rejected
// child's token is removed (Eq. e2 applied to all of them), from the pass's own
// draft-term sum minus those tokens' terms, computed the same way. Children
// are rejected in index order, so the running sum adds their terms in that
// order.
template <int kCap>
__device__ inline void update_remaining_mass(Lds<TreeSmem<kCap>>& sm, int j, int l,
                                             bool pass_summed_draft) {
  if (pass_summed_draft) {
    sm.sdsum[j] = sm.res_sd;
    sm.flags[j] |= kFlagSd;
  }
  const double total = sm.sdsum[j];
  const double removed = sm.removed[j] + sm.et[l];
  sm.removed[j] = removed;
  sm.rem[j] = (total - removed) / total;
}

template <int kCap>
__device__ inline void batch_begin(Lds<TreeSmem<kCap>>& sm, int cmd, int node) {
  sm.cmd = kCmdBatch;
  sm.bn = 1;
  sm.bnode[0] = static_cast<int16_t>(node);
  sm.bcmd[0] = static_cast<int8_t>(cmd);
  sm.cmd_ap = sm.cmd_bp = sm.cmd_cb = sm.cmd_cs = 0.0;
}

// Adds STATS of the internal nodes without statistics on the leftmost
// remaining path from c: the traversal descends through them next.
template <int kCap>
__device__ inline void batch_add_descent(Lds<TreeSmem<kCap>>& sm, int c) {
  while (sm.bn < kMaxBatch && sm.child_count[c] > 0 && sm.next_child[c] < sm.child_count[c]) {
    if (!(sm.flags[c] & kFlagStats)) {
      sm.bnode[sm.bn] = static_cast<int16_t>(c);
      sm.bcmd[sm.bn] = static_cast<int8_t>(kCmdStats2);
      ++sm.bn;
    }
    c = sm.child_list[sm.child_start[c] + sm.next_child[c]];
  }
}

// STATS of node j (two rows, or the target row of an accepted leaf); with
// `descent`, also of the internal nodes below j the traversal reaches next.
template <int kCap>
__device__ inline void issue_stats(Lds<TreeSmem<kCap>>& sm, int node, bool two, bool descent) {
  batch_begin(sm, two ? kCmdStats2 : kCmdStats1, node);
  if (descent && sm.next_child[node] < sm.child_count[node])
    batch_add_descent(sm, sm.child_list[sm.child_start[node] + sm.next_child[node]]);
}

// SPASS at j (a child of j was just rejected); with `descent`, also STATS of
// the internal nodes the traversal descends into after it: j's next child c
// and the leftmost path below it, if c's chain rate stays above zero. That
// rate is [A' r(c) - B']_+ with A' = alpha / S, B' = beta / S, so its sign is
// known before S is: it is positive iff alpha r(c) > beta.
template <int kCap>
__device__ inline void issue_spass(Lds<TreeSmem<kCap>>& sm, int node, double alpha, double beta,
                                   bool wo, bool descent) {
  batch_begin(sm, (wo && !(sm.flags[node] & kFlagSd)) ? kCmdSPassSd : kCmdSPass, node);
  sm.cmd_ap = alpha * sm.invsb[node];
  sm.cmd_bp = beta * sm.invss[node];
  sm.cmd_cb = sm.cb[node];
  sm.cmd_cs = sm.cs[node];
  if (descent && sm.next_child[node] < sm.child_count[node]) {
    const int c = sm.child_list[sm.child_start[node] + sm.next_child[node]];
    if (alpha * sm.r0[c] > beta) batch_add_descent(sm, c);
  }
}

template <int kCap>
__device__ inline void request_sample(Lds<TreeSmem<kCap>>& sm, bool from_stats, bool two,
                                      double ap, double bp, double cb, double cs) {
  sm.cmd = kCmdLocalSample;
  sm.smp_from_stats = from_stats ? 1 : 0;
  sm.smp_two = two ? 1 : 0;
  sm.smp_ap = ap;
  sm.smp_bp = bp;
  sm.smp_cb = cb;
  sm.smp_cs = cs;
}

template <int kCap>
__device__ inline void fail(Lds<TreeSmem<kCap>>& sm, int status) {
  sm.status = status;
  sm.cmd = kCmdDone;
}

template <int kCap>
__device__ inline void init_node_state(Lds<TreeSmem<kCap>>& sm, int c, double pi) {
  sm.pi[c] = pi;
  sm.A[c] = 1.0;
  sm.B[c] = 0.0;
  sm.rem[c] = 1.0;
  sm.removed[c] = 0.0;
}

struct TraversalArgs {
  int num_nodes, mode, algo, early;
};

struct Ctl {
  int phase, cur, accepted, rejected, rows, resid, tests, pinit_next;
  double alpha, beta;
};

// Runs until the next batch of passes or a local sample is needed, or the tree
// is done. `done_cmd` is the kind of pass 0 of the batch (or the local sample)
// whose result is in sm.res_*; STATS results are already in the node arrays.
template <int kCap>
__device__ __forceinline__ void advance_impl(Lds<TreeSmem<kCap>>& sm, TraversalArgs P,
                                             int done_cmd, Ctl& ct) {
  const bool summed_draft = done_cmd == kCmdSPassSd;
  const bool wo = P.mode == TV_SIBLINGS_WITHOUT_REPLACEMENT;
  const bool tv_algo = P.algo == static_cast<int>(tv::Algo::kTraversal);
  for (;;) {
    switch (ct.phase) {
      // ---- Alg. 3 initial chain rates for the p_init output -------------
      case kPhPinit: {
        // STATS of every node with children, up to a batch at a time
        int first = -1, n = 0;
        for (int j = ct.pinit_next; j < P.num_nodes; ++j) {
          if (sm.child_count[j] == 0 || (sm.flags[j] & kFlagStats)) continue;
          if (n == kMaxBatch) break;
          if (first < 0) {
            batch_begin(sm, kCmdStats2, j);
            first = j;
          } else {
            sm.bnode[sm.bn] = static_cast<int16_t>(j);
            sm.bcmd[sm.bn] = static_cast<int8_t>(kCmdStats2);
            ++sm.bn;
          }
          ++n;
        }
        if (n > 0) {
          ct.pinit_next = first;
          return;
        }
        for (int j = 0; j < P.num_nodes; ++j)
          if (sm.child_count[j] > 0 && (sm.flags[j] & kFlagBad)) {
            fail(sm, TV_TREE_NONFINITE);
            return;
          }
        sm.pini[0] = 1.0;
        for (int i = 1; i < P.num_nodes; ++i) {
          const int j = sm.parent[i];
          if (sm.pini[j] == 0.0) { sm.pini[i] = 0.0; continue; }
          sm.pini[i] = fmin(sm.pini[j] * sm.r0[i], 1.0);
        }
        ct.phase = tv_algo ? kPhDescend : kPhTlVisit;
        continue;
      }
      // ---- Traversal Verification ----------------------------------------
      case kPhDescend: {   // walk to the first leaf of the remaining tree
        const int j = ct.cur;
        if (sm.next_child[j] < sm.child_count[j] && sm.pi[j] == 0.0) {
          // every chain through j has rate 0: the remaining children and their
          // subtrees are pruned without visiting them (their outputs are
          // written when the tree finishes), and j itself is tested next
          sm.prune_from[j] = sm.next_child[j];
          sm.flags[j] |= kFlagPrunedBelow;
          sm.any_pruned = 1;
          sm.next_child[j] = static_cast<int16_t>(sm.child_count[j]);
          ct.phase = kPhTest;
          continue;
        }
        if (sm.next_child[j] < sm.child_count[j]) {
          if (sm.pi[j] > 0.0) {
            if (!(sm.flags[j] & kFlagConsulted)) {
              sm.flags[j] |= kFlagConsulted;
              ++ct.rows;
            }
            if (!(sm.flags[j] & kFlagStats)) { issue_stats(sm, j, true, true); return; }
            if (sm.flags[j] & kFlagBad) { fail(sm, TV_TREE_NONFINITE); return; }
          }
          const int c = sm.child_list[sm.child_start[j] + sm.next_child[j]];
          init_node_state(sm, c, child_rate(sm, P.mode, j, c));
          ct.cur = c;
          continue;
        }
        ct.phase = kPhTest;
        continue;
      }
      case kPhTest: {
        const int l = ct.cur;
        if (l == 0) {                       // only the root is left: p(X_0) = 1
          ct.accepted = 0;
          sm.state[0] = TV_NODE_ACCEPTED;
          ct.phase = kPhFinal;
          continue;
        }
        const int j = sm.parent[l];
        if (sm.pi[j] == 0.0) {              // parent can no longer be accepted
          sm.state[l] = TV_NODE_PRUNED;
          sm.theta[l] = 0.0f;
          ++sm.next_child[j];
          ct.cur = j;
          ct.phase = kPhDescend;
          continue;
        }
        const double th = sm.pi[l];
        sm.theta[l] = static_cast<float>(th);
        ++ct.tests;
        if (static_cast<double>(sm.u[l]) < th) {
          sm.state[l] = TV_NODE_ACCEPTED;
          ct.accepted = l;
          ct.phase = kPhFinal;
          continue;
        }
        sm.state[l] = TV_NODE_REJECTED;
        ++sm.next_child[j];
        if (P.early && j != 0 && sm.next_child[j] == sm.child_count[j] &&
            static_cast<double>(sm.u[j]) >= sm.pi[j]) {
          // Early rejection: l was j's last child and j is tested next. Eq. (e3)
          // never raises j's rate (S <= p by Eq. e1), so u[j] >= p already
          // rejects j, whatever the update would give; the update, which only
          // j's own test and a residual at j could use, is skipped. The test
          // below records the current p as theta (an upper bound), which is
          // why this applies only when theta is not an output.
          ct.cur = j;
          continue;
        }
        const double cc = wo ? 1.0 / sm.rem[j] : 1.0;
        ct.alpha = sm.pi[j] * sm.A[j];
        ct.beta = sm.pi[j] * sm.B[j] + cc;
        ct.rejected = l;
        ct.phase = kPhAfterSPass;
        issue_spass(sm, j, ct.alpha, ct.beta, wo, true);
        return;
      }
      case kPhAfterSPass: {                 // Eq. (e1), (e2), (e3) at the parent
        const int l = ct.rejected;
        const int j = sm.parent[l];
        const double S = sm.res_S;
        ++ct.resid;
        if (S > 0.0) {
          const double inv = 1.0 / S;
          sm.A[j] = ct.alpha * inv;
          sm.B[j] = ct.beta * inv;
          sm.pi[j] = S / (S + (1.0 - sm.pi[j]));
        } else if (j == 0) {
          fail(sm, TV_TREE_DEGENERATE);
          return;
        } else {
          sm.pi[j] = 0.0;
        }
        if (wo) update_remaining_mass(sm, j, l, summed_draft);
        ct.cur = j;
        ct.phase = kPhDescend;
        continue;
      }
      // ---- Token-level verification --------------------------------------
      case kPhTlVisit: {
        const int j = ct.cur;
        if (sm.child_count[j] == 0) {       // accepted leaf: Y from its target row
          ct.accepted = j;
          if (j == 0) sm.state[0] = TV_NODE_ACCEPTED;
          ct.phase = kPhFinal;
          continue;
        }
        if (!(sm.flags[j] & kFlagConsulted)) {
          sm.flags[j] |= kFlagConsulted;
          ++ct.rows;
        }
        if (!(sm.flags[j] & kFlagStats)) { issue_stats(sm, j, true, false); return; }
        if (sm.flags[j] & kFlagBad) { fail(sm, TV_TREE_NONFINITE); return; }
        if (sm.next_child[j] == sm.child_count[j]) {   // all rejected: Y from residual
          ct.accepted = j;
          if (j == 0) sm.state[0] = TV_NODE_ACCEPTED;
          ct.phase = kPhFinal;
          continue;
        }
        const int c = sm.child_list[sm.child_start[j] + sm.next_child[j]];
        const double th = child_rate(sm, P.mode, j, c);
        sm.theta[c] = static_cast<float>(th);
        ++ct.tests;
        if (static_cast<double>(sm.u[c]) < th) {
          sm.state[c] = TV_NODE_ACCEPTED;
          init_node_state(sm, c, 1.0);
          ct.cur = c;
          continue;
        }
        sm.state[c] = TV_NODE_REJECTED;
        ++sm.next_child[j];
        const double cc = wo ? 1.0 / sm.rem[j] : 1.0;
        ct.alpha = sm.A[j];
        ct.beta = sm.B[j] + cc;
        ct.rejected = c;
        ct.phase = kPhTlAfterSPass;
        issue_spass(sm, j, ct.alpha, ct.beta, wo, false);
        return;
      }
      case kPhTlAfterSPass: {               // Algorithm 2 rejection branch
        const int c = ct.rejected;
        const int j = sm.parent[c];
        const double S = sm.res_S;
        ++ct.resid;
        if (!(S > 0.0)) { fail(sm, TV_TREE_DEGENERATE); return; }
        const double inv = 1.0 / S;
        sm.A[j] = ct.alpha * inv;
        sm.B[j] = ct.beta * inv;
        if (wo) update_remaining_mass(sm, j, c, summed_draft);
        ct.phase = kPhTlVisit;
        continue;
      }
      // ---- Final sample Y --------------------------------------------------
      case kPhFinal: {
        const int a = ct.accepted;
        if (sm.child_count[a] == 0) {       // accepted leaf: its target row
          ct.phase = kPhFinalLeafStats;
          issue_stats(sm, a, false, false);
          return;
        }
        if (sm.spass_node == a) {           // weights of the SPASS just done at a
          ct.phase = kPhAfterSample;
          request_sample(sm, false, true, sm.last_ap, sm.last_bp, sm.last_cb, sm.last_cs);
          return;
        }
        ct.phase = kPhFinalWSum;            // residual weights need a pass of their own
        batch_begin(sm, kCmdWSum, a);
        sm.cmd_ap = sm.A[a] * sm.invsb[a];
        sm.cmd_bp = sm.B[a] * sm.invss[a];
        sm.cmd_cb = sm.cb[a];
        sm.cmd_cs = sm.cs[a];
        return;
      }
      case kPhFinalLeafStats: {
        const int a = ct.accepted;
        if (sm.flags[a] & kFlagBad) { fail(sm, TV_TREE_NONFINITE); return; }
        ct.phase = kPhAfterSample;
        request_sample(sm, true, false, 1.0, 0.0, sm.cb[a], 0.0);
        return;
      }
      case kPhFinalWSum: {
        ct.phase = kPhAfterSample;
        request_sample(sm, false, true, sm.last_ap, sm.last_bp, sm.last_cb, sm.last_cs);
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

// The controller's scalars live in registers for the duration of a step.
template <int kCap>
__device__ __attribute__((always_inline)) void advance(Lds<TreeSmem<kCap>>& sm, TraversalArgs P,
                                                      int done_cmd) {
  Ctl ct{sm.phase, sm.cur, sm.accepted, sm.rejected, sm.rows_consulted, sm.resid_passes,
         sm.tests, sm.pinit_next, sm.alpha, sm.beta};
  advance_impl(sm, P, done_cmd, ct);
  sm.phase = ct.phase;
  sm.cur = ct.cur;
  sm.accepted = ct.accepted;
  sm.rejected = ct.rejected;
  sm.rows_consulted = ct.rows;
  sm.resid_passes = ct.resid;
  sm.tests = ct.tests;
  sm.pinit_next = ct.pinit_next;
  sm.alpha = ct.alpha;
  sm.beta = ct.beta;
}

// ---------------------------------------------------------------------------
// Tree set-up and outputs
// ---------------------------------------------------------------------------

template <typename T, class PP>
__device__ __forceinline__ const T* row_ptr(const PP& P, const void* base, int b, int node) {
  return static_cast<const T*>(base) +
         (static_cast<size_t>(b) * P.num_nodes + node) * static_cast<size_t>(P.vocab);
}

// Loads and checks tree b into LDS, gathers every node's logits at its token
// in its parent's rows, and starts the traversal (all threads).
template <typename T, class A, int kCap>
__device__ __attribute__((noinline)) void begin_tree(Lds<TreeSmem<kCap>>& sm, Lds<WgScratch>& ws,
                                                     const Lds<Params>& P, A ar, int b) {
  constexpr int kPer = (kCap + kNT - 1) / kNT;   // nodes per thread
  const int tid = threadIdx.x;
  const int n1 = P.num_nodes;
  const int V = P.vocab;
  const size_t tree_off = static_cast<size_t>(b) * n1;
  if (tid == 0) sm.status = TV_TREE_OK;
  __syncthreads();
  // every load of the tree at once: links, tokens, uniforms, then each
  // node's parent logits at its token (at clamped indices, so that they stay
  // in the rows whatever the links; stored only once the tree is checked)
  int pr[kPer], xr[kPer];
  float ur[kPer], vb[kPer], vs[kPer];
#pragma unroll
  for (int t = 0; t < kPer; ++t) {
    const int i = tid + t * kNT;
    pr[t] = xr[t] = 0;
    ur[t] = 0.0f;
    if (i < n1) {
      pr[t] = P.parents[tree_off + i];
      xr[t] = P.tokens[tree_off + i];
      ur[t] = P.uniforms[tree_off + i];
    }
  }
  int bad_parent = 0, bad_token = 0;
#pragma unroll
  for (int t = 0; t < kPer; ++t) {
    const int i = tid + t * kNT;
    vb[t] = vs[t] = 0.0f;
    if (i < n1) {
      const int p = pr[t], x = xr[t];
      if (i == 0 ? p != -1 : (p < 0 || p >= i)) bad_parent = 1;
      if (i > 0 && (x < 0 || x >= V)) bad_token = 1;
      const int pc = (i == 0 || p < 0 || p >= i) ? 0 : p;
      if (i > 0) {
        const int xc = min(max(x, 0), V - 1);
        vb[t] = Elem<T>::scalar(row_ptr<T>(P, P.target, b, pc) + xc);
        vs[t] = Elem<T>::scalar(row_ptr<T>(P, P.draft, b, pc) + xc);
      }
      sm.parent[i] = static_cast<int16_t>(i == 0 ? -1 : pc);
      sm.token[i] = x;
      sm.u[i] = ur[t];
      sm.child_count[i] = 0;
      sm.next_child[i] = 0;
      sm.state[i] = TV_NODE_UNTESTED;
      sm.flags[i] = 0;
      sm.theta[i] = -1.0f;
      sm.pini[i] = -1.0;
    }
  }
  bad_parent = __syncthreads_or(bad_parent);
  bad_token = __syncthreads_or(bad_token);
  if (tid == 0) {
    if (bad_parent) sm.status = TV_TREE_BAD_PARENT;
    else if (bad_token) sm.status = TV_TREE_BAD_TOKEN;
  }
  __syncthreads();
  if (sm.status == TV_TREE_OK) {
    for (int i = 1 + tid; i < n1; i += kNT)
      __hip_atomic_fetch_add(&sm.child_count[sm.parent[i]], 1, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_WORKGROUP);
    __syncthreads();
    {
      // first child slot of every node: exclusive prefix sum of the counts,
      // thread t summing the nodes [t q, t q + q)
      const int q = (n1 + kNT - 1) / kNT;
      const int lo = min(n1, tid * q), hi = min(n1, lo + q);
      int loc = 0;
      for (int j = lo; j < hi; ++j) loc += sm.child_count[j];
      int run = static_cast<int>(block_incl_scan(ws, static_cast<double>(loc))) - loc;
      for (int j = lo; j < hi; ++j) {
        sm.child_start[j] = static_cast<int16_t>(run);
        run += sm.child_count[j];
      }
    }
    __syncthreads();
    // the children in any order (the counts, counted down, hand out the
    // slots), then the counts again from the starts
    for (int i = 1 + tid; i < n1; i += kNT) {
      const int p = sm.parent[i];
      const int pos = __hip_atomic_fetch_add(&sm.child_count[p], -1, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_WORKGROUP) - 1;
      sm.child_list[sm.child_start[p] + pos] = static_cast<int16_t>(i);
    }
    __syncthreads();
    for (int j = tid; j < n1; j += kNT)
      sm.child_count[j] = (j + 1 < n1 ? sm.child_start[j + 1] : n1 - 1) - sm.child_start[j];
    __syncthreads();
    // a child's rank is the number of its siblings with smaller indices; the
    // same scan finds a token drawn twice among siblings
    const bool wo = P.mode == TV_SIBLINGS_WITHOUT_REPLACEMENT;
    int rk[kPer];
    int dup = 0;
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int i = 1 + tid + t * kNT;
      rk[t] = 0;
      if (i < n1) {
        const int p = sm.parent[i], s0 = sm.child_start[p], cnt = sm.child_count[p];
        const int x = sm.token[i];
        int r = 0;
        for (int k2 = 0; k2 < cnt; ++k2) {
          const int c = sm.child_list[s0 + k2];
          const int xc = sm.token[c];
          r += c < i;
          dup |= static_cast<int>(wo & (c != i) & (xc == x));
        }
        rk[t] = r;
      }
    }
    __syncthreads();
    // in index order
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int i = 1 + tid + t * kNT;
      if (i < n1) {
        sm.child_list[sm.child_start[sm.parent[i]] + rk[t]] = static_cast<int16_t>(i);
        sm.rank[i] = static_cast<int16_t>(rk[t]);
      }
    }
    dup = __syncthreads_or(dup);
    if (tid == 0 && dup) sm.status = TV_TREE_DUP_SIBLING;
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int i = tid + t * kNT;
      if (i > 0 && i < n1) {
        sm.gb[i] = vb[t];
        sm.gs[i] = vs[t];
      }
    }
    if (P.tmax) {
      // Row statistics given by the caller: every node with children has its
      // STATS results (the frame of its maximum and the inverse of its sum),
      // so the traversal issues no STATS pass; then every child's ratio.
      for (int j = tid; j < n1; j += kNT) {
        if (sm.child_count[j] == 0) continue;
        const float mb = P.tmax[tree_off + j], ms = P.dmax[tree_off + j];
        const double tb = P.tsum[tree_off + j], ts = P.dsum[tree_off + j];
        const bool bad = !(mb > -INFINITY) || !isfinite(mb) || !(ms > -INFINITY) ||
                         !isfinite(ms) || !(tb > 0.0) || !isfinite(tb) || !(ts > 0.0) ||
                         !isfinite(ts);
        sm.cb[j] = ar.frame(bad ? 0.0f : mb);
        sm.cs[j] = ar.frame(bad ? 0.0f : ms);
        sm.invsb[j] = bad ? 1.0 : 1.0 / (tb * ar.frame_rounding(mb));
        sm.invss[j] = bad ? 1.0 : 1.0 / (ts * ar.frame_rounding(ms));
        sm.flags[j] |= kFlagStats | (bad ? kFlagBad : 0);
      }
      __syncthreads();
      for (int c = 1 + tid; c < n1; c += kNT) child_ratio(sm, ar, sm.parent[c], c);
    }
  }
  if (tid == 0) {
    sm.has_tree = 1;
    sm.tree = b;
    sm.cur = 0;
    sm.accepted = -1;
    sm.rows_consulted = sm.resid_passes = sm.tests = 0;
    sm.pinit_next = 0;
    sm.any_pruned = 0;
    init_node_state(sm, 0, 1.0);
    sm.res_y = -1;
    sm.cmd = kCmdNone;
    sm.pending = 0;
    sm.spass_node = -1;
    const bool tv_algo = P.algo == static_cast<int>(tv::Algo::kTraversal);
    if (P.p_init && tv_algo) sm.phase = kPhPinit;
    else sm.phase = tv_algo ? kPhDescend : kPhTlVisit;
  }
  __syncthreads();
}

// Writes the tree's outputs (all threads of one member).
template <int kCap>
__device__ __attribute__((always_inline)) void finish_tree(Lds<TreeSmem<kCap>>& sm,
                                                           const Lds<Params>& P) {
  const int tid = threadIdx.x;
  const int b = sm.tree;
  const int n1 = P.num_nodes;
  const size_t tree_off = static_cast<size_t>(b) * n1;
  const bool ok = sm.status == TV_TREE_OK;
  // the accepted node's depth (thread 0 walks to the root meanwhile)
  int depth = 0;
  if (tid == 0 && ok)
    for (int x = sm.accepted; x > 0; x = sm.parent[x]) ++depth;
  // Nodes below a chain of rate 0 that the traversal skipped. The edge into
  // node x is cut if x's parent is pruned below at or before x's rank; a node
  // is pruned if an edge on its path to the root is cut. Pointer jumping:
  // every node holds the OR of the cuts from itself up to (not including) its
  // current ancestor, and each round doubles that span, so the rounds number
  // log2 of the depth. prune_from and next_child, which the finished
  // traversal no longer reads, hold the spans' cut flags and ancestors.
  if (sm.any_pruned) {
    constexpr int kPer = (kCap + kNT - 1) / kNT;
    int anc[kPer], cut[kPer];
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int i = tid + t * kNT;
      const bool in = i > 0 && i < n1;
      const int p = in ? sm.parent[i] : 0;
      // no short-circuit: a branch per condition would serialise the reads
      const int f = sm.flags[p], ri = sm.rank[in ? i : 0], pf = sm.prune_from[p];
      cut[t] = static_cast<int>(in & ((f & kFlagPrunedBelow) != 0) & (ri >= pf));
      anc[t] = p;
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int i = tid + t * kNT;
      if (i < n1) {
        sm.prune_from[i] = static_cast<int16_t>(cut[t]);
        sm.next_child[i] = static_cast<int16_t>(anc[t]);
      }
    }
    __syncthreads();
    for (;;) {
      int fa[kPer], aa[kPer];
#pragma unroll
      for (int t = 0; t < kPer; ++t) {
        fa[t] = sm.prune_from[anc[t]];
        aa[t] = sm.next_child[anc[t]];
      }
      __syncthreads();
      int live = 0;
#pragma unroll
      for (int t = 0; t < kPer; ++t) {
        const int i = tid + t * kNT;
        cut[t] |= fa[t];
        anc[t] = aa[t];
        live |= anc[t];
        if (i < n1) {
          sm.prune_from[i] = static_cast<int16_t>(cut[t]);
          sm.next_child[i] = static_cast<int16_t>(anc[t]);
        }
      }
      if (!__syncthreads_or(live)) break;
    }
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int i = tid + t * kNT;
      if (cut[t] && i < n1 && sm.state[i] == TV_NODE_UNTESTED) {
        sm.state[i] = TV_NODE_PRUNED;
        sm.theta[i] = 0.0f;
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < n1; i += kNT) {
    if (P.node_state) P.node_state[tree_off + i] = ok ? static_cast<int8_t>(sm.state[i]) : 0;
    if (P.node_theta) P.node_theta[tree_off + i] = ok ? sm.theta[i] : -1.0f;
    if (P.p_init) P.p_init[tree_off + i] = ok ? static_cast<float>(sm.pini[i]) : -1.0f;
  }
  if (tid == 0) {
    P.status[b] = sm.status;
    P.accept_len[b] = ok ? depth : -1;
    P.accepted_node[b] = ok ? sm.accepted : -1;
    P.bonus_token[b] = ok ? sm.res_y : -1;
    if (P.counters) {
      int32_t* c = P.counters + static_cast<size_t>(b) * TV_NUM_COUNTERS;
      c[0] = ok ? sm.rows_consulted : 0;
      c[1] = ok ? sm.resid_passes : 0;
      c[2] = ok ? (sm.child_count[sm.accepted] == 0 ? 1 : 0) : 0;
      c[3] = ok ? sm.tests : 0;
    }
    sm.has_tree = 0;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Group exchange: combining the members' partials, the local sample
// ---------------------------------------------------------------------------

// Loads member `lane`'s partial of one pass until all four words carry the
// batch's tag (all lanes < G of the wave). Returns false if the launch was
// abandoned meanwhile (the wait limit passed here or elsewhere).
template <class PP>
__device__ __forceinline__ bool await_part(const PP& P, const SegPart* part, int G,
                                           uint64_t tag, uint64_t (&w)[4]) {
  const int lane = threadIdx.x & 63;
  const long long t0 = wall_clock64();
  for (int it = 0;; ++it) {
    bool ok = true;
    if (lane < G) {
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = ld_rlx(&part[lane].w[j]);
    }
    // with the loads, this wave's stores of the last batch's partials are
    // performed (the order the exchange relies on)
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    if (lane < G) ok = tags_are(w, tag);
    if (__ballot(!ok) == 0) return true;
    // the abort flag and the clock are checked every 16th failed poll (every
    // failed poll with a wait limit of 0)
    if ((it & 15) == 15 || P.spin_limit == 0) {
      uint32_t ab = 0;
      if (lane == 0) ab = ld_rlx(ws_abort(P));
      if (__shfl(ab, 0, 64)) return false;
      if (wall_clock64() - t0 >= P.spin_limit) {
        if (lane == 0) st_rlx(ws_abort(P), 1u);
        return false;
      }
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// Child c's original ratio r0 = p(x)/q(x) at its parent j and its draft term,
// from j's row statistics and the gathered logits; a drafted token the draft
// cannot produce (draft logit -inf) marks j bad.
template <class A, int kCap>
__device__ __forceinline__ void child_ratio(Lds<TreeSmem<kCap>>& sm, const A& ar, int j, int c) {
  const double kd = ar.kd();
  const double Cb = sm.cb[j], Cs = sm.cs[j];
  const double norm = sm.invsb[j] / sm.invss[j];   // ts / tb
  const double lp = fma(static_cast<double>(sm.gb[c]), kd, Cb);
  const double lq = fma(static_cast<double>(sm.gs[c]), kd, Cs);
  sm.r0[c] = exp2(lp - lq) * norm;
  sm.et[c] = ar.ex(sm.gs[c], Cs);
  if (sm.gs[c] == -INFINITY) sm.flags[j] |= kFlagBad;
}

// Combines the members' partials of the completed batch (all threads): wave w
// waits for and takes passes w, w + 4, lanes are members; STATS results go to
// the node arrays, a SPASS / WSUM result to res_S / res_sd. Returns false if
// the launch was abandoned.
template <typename T, class A, int kCap>
__device__ __attribute__((always_inline)) bool combine(Lds<TreeSmem<kCap>>& sm,
                                                       Lds<WgScratch>& ws,
                                                       const Lds<Params>& P, A ar, int g) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bn = sm.bn;
  const int G = sm.geff;                // contributors of this batch
  const int par = static_cast<int>(sm.seq & 1u);
  const uint64_t tag = batch_tag(sm.seq);
  if (tid == 0) ws.stop = 0;
  __syncthreads();
  for (int p = wave; p < bn; p += kNW) {
    const int cmd = sm.bcmd[p];
    const int node = sm.bnode[p];
    const SegPart* part = ws_parts(P, g, par, p);
    uint64_t w[4] = {0, 0, 0, 0};
    if (!await_part(P, part, G, tag, w)) {
      if (lane == 0) ws.stop = 1;
      break;
    }
    double s0 = 0.0, s1 = 0.0;
    float m0 = -INFINITY, m1 = -INFINITY;
    if (lane < G) {
      s0 = dec_sum(w[0]);
      s1 = dec_sum(w[1]);
      m0 = dec_max(w[2]);
      m1 = dec_max(w[3]);
    }
    if (p == 0 && lane == 0) ws.hnext = max_count(w[3]);   // member 0's report
    if (cmd == kCmdStats2 || cmd == kCmdStats1) {
      const bool two = cmd == kCmdStats2;
      const float Mb = wave_max(m0);
      const float Ms = two ? wave_max(m1) : -INFINITY;
      const double Cb = ar.frame(Mb);
      const double Cs = two ? ar.frame(Ms) : 0.0;
      // stripe sums in the row's frame; a stripe with no finite value adds 0 (or NaN)
      double tb = (m0 > -INFINITY) ? s0 * exp2(Cb - ar.frame(m0)) : s0;
      double ts = two ? ((m1 > -INFINITY) ? s1 * exp2(Cs - ar.frame(m1)) : s1) : 0.0;
      tb = __shfl(wave_sum(tb), 0, 64);
      ts = __shfl(wave_sum(ts), 0, 64);
      if (lane == 0) {
        const bool bad = !(Mb > -INFINITY) || !isfinite(tb) ||
                         (two && (!(Ms > -INFINITY) || !isfinite(ts)));
        sm.cb[node] = Cb;
        sm.invsb[node] = 1.0 / tb;
        if (two) {
          sm.cs[node] = Cs;
          sm.invss[node] = 1.0 / ts;
        }
        sm.flags[node] |= kFlagStats | (bad ? kFlagBad : 0);
      }
    } else {
      const double S = __shfl(wave_sum(s0), 0, 64);
      const double sd = __shfl(wave_sum(s1), 0, 64);
      if (lane == 0) {
        sm.res_S = S;
        sm.res_sd = sd;
      }
    }
  }
  __syncthreads();
  if (ws.stop) return false;
  if (tid == 0) {
    sm.geff_last = G;
    const int next = P.G + ws.hnext;
    sm.geff = next > G ? next : G;
  }
  // children's original ratios r0 = p(x)/q(x) and draft terms: 32 threads per
  // pass (a node with bad statistics gets values it never uses: the traversal
  // fails the tree before it reads them)
  static_assert(kMaxBatch * 32 <= kNT, "one thread group of 32 per pass");
  if (tid < bn * 32) {
    const int p = tid >> 5;
    const int node = sm.bnode[p];
    if (sm.bcmd[p] == kCmdStats2)
      for (int i = tid & 31; i < sm.child_count[node]; i += 32)
        child_ratio(sm, ar, node, sm.child_list[sm.child_start[node] + i]);
  }
  __syncthreads();
  return true;
}

// Inverse-CDF draw of Y (all threads of one member). The weights of the
// stripes come from the partials of pass 0 of the batch just completed; the
// stripe holding u*W is rescanned. Its units (head elements, 16-byte vectors,
// tail elements, in token order) are summed in chunks of 64 consecutive units,
// one unit per lane, with many chunks' loads in flight per wave; a scan over
// the chunk sums finds the chunk, a wave scan over its units the unit, and the
// lane holding that unit finds the token.
constexpr int kSampleChunks = 256;      // chunk sums held at once (a window)
constexpr int kSampleInFlight = 4;      // chunks per wave whose loads are in flight

template <typename T, class A, int kCap>
__device__ __attribute__((noinline)) void local_sample(Lds<TreeSmem<kCap>>& sm, Lds<WgScratch>& ws,
                                                       const Lds<Params>& P, A ar, int g) {
  constexpr int E = Elem<T>::E;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int node = sm.bnode[0];
  const int G = sm.geff_last;           // contributors of the batch just completed
  if (tid < 64) {
    const SegPart* part = ws_parts(P, g, static_cast<int>(sm.seq & 1u), 0);
    double w = 0.0;
    if (lane < G) {
      // the combine has seen this batch's tags in every word
      const double s0 = dec_sum(ld_rlx(&part[lane].w[0]));
      if (sm.smp_from_stats) {
        const float m0 = dec_max(ld_rlx(&part[lane].w[2]));
        w = (m0 > -INFINITY) ? s0 * exp2(sm.smp_cb - ar.frame(m0)) : 0.0;
      } else {
        w = s0;
      }
    }
    double incl = w;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double o = __shfl_up(incl, off, 64);
      if (lane >= off) incl += o;
    }
    const double W = __shfl(incl, G - 1, 64);
    const double target = static_cast<double>(sm.u[0]) * W;
    const uint64_t pos = __ballot(lane < G && w > 0.0);
    const uint64_t hits = __ballot(lane < G && w > 0.0 && target < incl);
    int seg = -1;
    bool fallback = false;
    if (W > 0.0 && isfinite(W) && pos != 0) {
      if (hits) {
        seg = __ffsll(static_cast<long long>(hits)) - 1;
      } else {                              // rounding at the end: last stripe with mass
        seg = 63 - __clzll(static_cast<long long>(pos));
        fallback = true;
      }
    }
    if (lane == 0) {
      ws.smp_seg = seg;
      ws.smp_chunk = -1;
      ws.smp_last_chunk = -1;
    }
    if (seg >= 0 && lane == seg) ws.smp_target = fallback ? INFINITY : target - (incl - w);
  }
  if (tid == 0) sm.res_y = -2;
  __syncthreads();
  const int seg = ws.smp_seg;
  if (seg < 0) return;     // no mass: res_y stays negative (degenerate)
  const T* rb = row_ptr<T>(P, P.target, sm.tree, node);
  const T* rs = row_ptr<T>(P, P.draft, sm.tree, node);
  const Geom geo = row_geom(rb, P.vocab);
  const SegRange r = stripe(geo, seg, G);
  const int nh = r.first ? geo.head : 0;
  const int nv = max(0, r.ve - r.vb);
  const int nt = r.last ? geo.tail : 0;
  const int nu = nh + nv + nt;
  const int tail0 = geo.head + geo.nvec * E;
  const TermParams tp{sm.smp_cb, sm.smp_cs, sm.smp_ap, sm.smp_bp};
  auto run = [&](auto two_tag) {
    constexpr bool TWO = decltype(two_tag)::value;
    using TM = Terms<A, TWO, false>;
    const TM tm(ar, tp);
    double unused = 0.0;
    // loads of unit i, unconditional: vectors clamped into the stripe (a
    // stripe without vectors reads a dummy vector of the workspace); head /
    // tail units are single elements read in unit_sum itself
    const bool has_vec = nv > 0;
    const T* lrb = has_vec ? rb : reinterpret_cast<const T*>(P.ws);
    const T* lrs = has_vec ? rs : reinterpret_cast<const T*>(P.ws);
    const int lhead = has_vec ? geo.head : 0;
    const int lvb = has_vec ? r.vb : 0, lvl = has_vec ? r.ve - 1 : 0;
    auto load_unit = [&](int i, uint4& vb, uint4& vs) {
      const int v = min(max(lvb + (i - nh), lvb), lvl);
      vb = load16(lrb, lhead, v);
      vs = TWO ? load16(lrs, lhead, v) : make_uint4(0, 0, 0, 0);
    };
    // sum of unit i: the same value wherever it is computed
    auto unit_sum = [&](int i, const uint4& vb, const uint4& vs) -> double {
      if (i >= nu) return 0.0;
      if (i < nh || i >= nh + nv) {
        const int x = i < nh ? i : tail0 + (i - nh - nv);
        return scalar_weight<T, TM, TWO>(tm, rb, rs, x, unused);
      }
      return vec_sum<T, TM, TWO>(tm, vb, vs, unused);
    };
    double running = 0.0;     // mass of the windows before this one
    double local = ws.smp_target;
    for (int w0 = 0; w0 < nu; w0 += kSampleChunks * 64) {
      const int nck = min(kSampleChunks, (nu - w0 + 63) / 64);
      // chunk sums: wave w takes chunks w, w + 4, ..., kSampleInFlight at a time
      for (int c0 = wave; c0 < nck; c0 += kNW * kSampleInFlight) {
        uint4 lb[kSampleInFlight], ls[kSampleInFlight];
#pragma unroll
        for (int j = 0; j < kSampleInFlight; ++j)
          load_unit(w0 + (c0 + j * kNW) * 64 + lane, lb[j], ls[j]);
#pragma unroll
        for (int j = 0; j < kSampleInFlight; ++j) {
          pin(lb[j]);
          pin(ls[j]);
        }
#pragma unroll
        for (int j = 0; j < kSampleInFlight; ++j) {
          const int c = c0 + j * kNW;
          if (c < nck) {
            const double s = wave_sum(unit_sum(w0 + c * 64 + lane, lb[j], ls[j]));
            if (lane == 0) ws.smp_chunks[c] = s;
          }
        }
      }
      __syncthreads();
      // the chunk holding the target: lane l of wave 0 scans chunks 4l .. 4l + 3
      if (tid < 64) {
        double cs[4], tot = 0.0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = 4 * lane + j;
          cs[j] = c < nck ? ws.smp_chunks[c] : 0.0;
          tot += cs[j];
        }
        double incl = tot;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const double o = __shfl_up(incl, off, 64);
          if (lane >= off) incl += o;
        }
        double before = running + (incl - tot);
        int hit = -1, lastpos = -1;
        double hit_target = 0.0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (cs[j] > 0.0) {
            lastpos = 4 * lane + j;
            if (hit < 0 && local < before + cs[j]) {
              hit = 4 * lane + j;
              hit_target = local - before;
            }
          }
          before += cs[j];
        }
        const uint64_t hits = __ballot(hit >= 0);
        const uint64_t poss = __ballot(lastpos >= 0);
        if (hits) {
          const int l = __ffsll(static_cast<long long>(hits)) - 1;
          if (lane == l) {
            ws.smp_chunk = w0 / 64 + hit;
            ws.smp_target = hit_target;
          }
        } else if (poss) {
          const int l = 63 - __clzll(static_cast<long long>(poss));
          if (lane == l) ws.smp_last_chunk = w0 / 64 + lastpos;
        }
        if (lane == 63) ws.smp_window = incl;   // mass of this window
      }
      __syncthreads();
      if (ws.smp_chunk >= 0) break;
      running += ws.smp_window;
    }
    // rounding at the end: the last chunk with mass, and in it the last
    // positive weight
    const bool fallback = ws.smp_chunk < 0;
    const int chunk = fallback ? ws.smp_last_chunk : ws.smp_chunk;
    if (chunk < 0) return;    // no positive weight: degenerate
    if (tid < 64) {
      const int i = chunk * 64 + lane;
      uint4 vb, vs;
      load_unit(i, vb, vs);
      const double us = unit_sum(i, vb, vs);
      double incl = us;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const double o = __shfl_up(incl, off, 64);
        if (lane >= off) incl += o;
      }
      const double tgt = fallback ? INFINITY : ws.smp_target;
      const uint64_t hits = __ballot(us > 0.0 && tgt < incl);
      const uint64_t poss = __ballot(us > 0.0);
      int pick = -1;
      bool last_of_unit = fallback;
      if (hits) {
        pick = __ffsll(static_cast<long long>(hits)) - 1;
      } else if (poss) {                    // rounding at the end: last unit with mass
        pick = 63 - __clzll(static_cast<long long>(poss));
        last_of_unit = true;
      }
      if (pick >= 0 && lane == pick) {
        double wd[E];
        int tok0 = 0, n = 1;
        if (i < nh || i >= nh + nv) {
          const int x = i < nh ? i : tail0 + (i - nh - nv);
          wd[0] = scalar_weight<T, TM, TWO>(tm, rb, rs, x, unused);
          tok0 = x;
        } else {
          float xb[E], xs[E];
          Elem<T>::unpack(vb, xb);
          if constexpr (TWO) {
            Elem<T>::unpack(vs, xs);
          } else {
#pragma unroll
            for (int e = 0; e < E; ++e) xs[e] = 0.0f;
          }
          typename TM::W wv[E];
          tm.weights(xb, xs, wv, unused);
#pragma unroll
          for (int e = 0; e < E; ++e) wd[e] = static_cast<double>(wv[e]);
          tok0 = geo.head + (r.vb + (i - nh)) * E;
          n = E;
        }
        double C = incl - us;
        int y = -1, last = -1;
#pragma unroll
        for (int e = 0; e < E; ++e) {     // unrolled: wd stays in registers
          if (e < n) {
            if (wd[e] > 0.0) {
              last = tok0 + e;
              if (!last_of_unit && y < 0 && tgt < C + wd[e]) y = tok0 + e;
            }
            C += wd[e];
          }
        }
        sm.res_y = y >= 0 ? y : last;    // rounding inside the unit: its last positive weight
      }
    }
  };
  if (sm.smp_two) run(std::true_type{});
  else run(std::false_type{});
  __syncthreads();
}

// One controller step (all threads; every member of the group runs it on the
// same data): publish this member's partials of the completed batch, combine
// everyone's, then advance the traversal until it needs the next batch, a
// local sample or the tree is done. With `after_sample`, only advance past the
// local sample just drawn (member 0 draws Y; the caller runs the sample, so
// that this function makes no call and keeps its return address in place).
// The partials are stored here rather than at the end of the batch: a call
// first waits for every memory access in flight, and stores issued inside it
// are awaited together with the first poll of the combine instead.
template <typename T, class A, int kCap>
__device__ __attribute__((noinline)) void controller_step(Lds<TreeSmem<kCap>>& sm,
                                                          Lds<WgScratch>& ws,
                                                          const Lds<Params>& P, A ar, int g,
                                                          int m, bool after_sample) {
  const int tid = threadIdx.x;
  if (sm.status == TV_TREE_OK) {
    int done_cmd = after_sample ? kCmdLocalSample : kCmdNone;
    if (!after_sample && sm.pending) {
      if (tid == 0) write_parts(P, ws, g, sm.seq, sm.bn, m, ws.res_count);
      if (!combine<T, A>(sm, ws, P, ar, g)) {   // the launch was abandoned
        if (tid == 0) sm.cmd = kCmdAbandon;
        __syncthreads();
        return;
      }
      done_cmd = sm.bcmd[0];
      if (tid == 0) sm.pending = 0;
    }
    if (tid == 0) {
      __builtin_amdgcn_s_setprio(3);
      advance(sm, TraversalArgs{P.num_nodes, P.mode, P.algo, P.early}, done_cmd);
      __builtin_amdgcn_s_setprio(0);
    }
  } else if (tid == 0) {
    sm.cmd = kCmdDone;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Helpers. A workgroup whose group has no tree left helps a running group: it
// takes a number in the group's helper count and then computes stripes of the
// group's passes like a member. Member 0 reads the count in every batch and
// reports it (capped at Gx - G) in its partial of pass 0, so every member
// agrees on the contributors of the next batch; the number only grows, and a
// helper once counted works in every later batch of that group. While the
// group has helpers, member 0 publishes each batch in a descriptor of 13
// 64-bit words, each holding the batch number in its high half, so a helper
// knows it read one whole descriptor when all 13 numbers agree.
// ---------------------------------------------------------------------------

constexpr int kDescWords = 16;     // per group: 13 descriptor words, word 15 the helper count

template <class PP>
__device__ __forceinline__ uint64_t* ws_desc(const PP& P, int g) {
  return reinterpret_cast<uint64_t*>(P.ws + P.off_desc) + static_cast<size_t>(g) * kDescWords;
}
template <class PP>
__device__ __forceinline__ uint32_t* ws_hcount(const PP& P, int g) {
  return reinterpret_cast<uint32_t*>(ws_desc(P, g) + 15);
}

constexpr uint32_t kDescDone = 1u << 31;

// Member 0, thread 0: publishes batch `seq` of the tree in sm for helpers.
template <int kCap>
__device__ __forceinline__ void publish_batch(const Params& P, int g, uint32_t seq,
                                              const Lds<TreeSmem<kCap>>& sm, int geff) {
  uint64_t* d = ws_desc(P, g);
  const uint64_t hi = static_cast<uint64_t>(seq) << 32;
  const uint32_t w0 = static_cast<uint32_t>(sm.tree) | (static_cast<uint32_t>(sm.bn) << 20) |
                      (static_cast<uint32_t>(geff) << 24);
  st_rlx(&d[0], hi | w0);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    uint32_t v = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int p = 2 * k + h;
      const uint32_t e = p < sm.bn ? (static_cast<uint32_t>(sm.bnode[p]) & 0x7FFu) |
                                         ((static_cast<uint32_t>(sm.bcmd[p]) & 0xFu) << 11)
                                   : 0u;
      v |= e << (16 * h);
    }
    st_rlx(&d[1 + k], hi | v);
  }
  const double prm[4] = {sm.cmd_ap, sm.cmd_bp, sm.cmd_cb, sm.cmd_cs};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint64_t b = static_cast<uint64_t>(__double_as_longlong(prm[k]));
    st_rlx(&d[5 + 2 * k], hi | (b & 0xFFFFFFFFull));
    st_rlx(&d[6 + 2 * k], hi | (b >> 32));
  }
}

// Member 0, thread 0: the group has no tree left.
template <class PP>
__device__ __forceinline__ void publish_done(const PP& P, int g, uint32_t seq) {
  st_rlx(&ws_desc(P, g)[0], (static_cast<uint64_t>(seq) << 32) | kDescDone);
}

// One pass of a stripe (all threads): STATS, or SPASS / WSUM weights.
template <typename T, class A, bool kShort>
__device__ __forceinline__ StripeResult stripe_pass(Lds<WgScratch>& ws, const T* rb, const T* rs,
                                                    const Geom& geo, const SegRange& r, int cmd,
                                                    const TermParams& tp, const A& ar) {
  StripeResult part;
  switch (cmd) {
    case kCmdStats2: stripe_stats<T, A, true, kShort>(ws, rb, rs, geo, r, ar, part); break;
    case kCmdStats1: stripe_stats<T, A, false, kShort>(ws, rb, rs, geo, r, ar, part); break;
    default:
      if (cmd == kCmdSPassSd) stripe_wsum<T, A, true, kShort>(ws, rb, rs, geo, r, ar, tp, part);
      else stripe_wsum<T, A, false, kShort>(ws, rb, rs, geo, r, ar, tp, part);
      break;
  }
  return part;
}

// Thread 0: writes contributor c's partials of batch `seq` (pass p's result
// for p < bn), together at the end of the batch, so that no store is in
// flight while the stripes run (the combine needs every pass anyway). One
// entry p >= bn, chosen in turn, gets an empty partial, so that no entry is
// more than 14 batches old: an entry left from an earlier batch never carries
// the tag of the batch being read.
template <class PP>
__device__ __forceinline__ void write_part(const PP& P, int g, uint32_t seq, int p, int c,
                                           const StripeResult& r, uint64_t count) {
  const uint64_t tag = batch_tag(seq);
  SegPart* dst = ws_parts(P, g, static_cast<int>(seq & 1u), p) + c;
  st_rlx(&dst->w[0], enc_sum(r.s0, tag));
  st_rlx(&dst->w[1], enc_sum(r.s1, tag));
  st_rlx(&dst->w[2], enc_max(r.m0, tag));
  st_rlx(&dst->w[3], enc_max(r.m1, tag, count));
}
template <class PP>
__device__ __forceinline__ void write_parts(const PP& P, const Lds<WgScratch>& ws, int g,
                                            uint32_t seq, int bn, int c, uint64_t count0) {
  for (int p = 0; p < bn; ++p) {
    const StripeResult r{ws.res[p].s0, ws.res[p].s1, ws.res[p].m0, ws.res[p].m1};
    write_part(P, g, seq, p, c, r, p == 0 ? count0 : 0);
  }
  const int pd = 1 + static_cast<int>((seq >> 1) % (kMaxBatch - 1));
  if (pd >= bn) write_part(P, g, seq, pd, c, StripeResult{0.0, 0.0, 0.0f, 0.0f}, 0);
  // The stores are not awaited here: the wave's next wait for a load of the
  // exchange (the combine's or a helper's first poll) waits for them too, and
  // it comes before any store of the next batch.
}

// Waits (wave 0) for a descriptor of group g newer than `last`, or its end,
// and copies it to LDS. ws.help_state: 0 new batch, 1 group done, 2 abandoned.
__device__ __forceinline__ void await_desc(Lds<WgScratch>& ws, const Params& P, int g,
                                           uint32_t last) {
  const int lane = threadIdx.x & 63;
  const uint64_t* d = ws_desc(P, g);
  const long long t0 = wall_clock64();
  for (int it = 0;; ++it) {
    const uint64_t w = lane < 13 ? ld_rlx(&d[lane]) : 0;
    // with the loads, this wave's stores of the last batch's partials are
    // performed (the order the exchange relies on)
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    const uint64_t w0 = __shfl(w, 0, 64);
    const uint32_t seq0 = static_cast<uint32_t>(w0 >> 32);
    if (static_cast<uint32_t>(w0) & kDescDone) {
      if (lane == 0) ws.help_state = 1;
      return;
    }
    const bool same = lane >= 13 || static_cast<uint32_t>(w >> 32) == seq0;
    if (__ballot(!same) == 0 && seq0 != last && seq0 != 0) {
      const uint32_t lo = static_cast<uint32_t>(w);
      if (lane == 0) {
        ws.d_seq = seq0;
        ws.d_tree = static_cast<int>(lo & 0xFFFFFu);
        ws.d_bn = static_cast<int>((lo >> 20) & 0xFu);
        ws.d_geff = static_cast<int>((lo >> 24) & 0x7Fu);
        ws.help_state = 0;
      }
      if (lane >= 1 && lane <= 4) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t e = (lo >> (16 * h)) & 0xFFFFu;
          ws.d_node[2 * (lane - 1) + h] = static_cast<int16_t>(e & 0x7FFu);
          ws.d_cmd[2 * (lane - 1) + h] = static_cast<int8_t>((e >> 11) & 0xFu);
        }
      }
      // parameters: lanes 5..12 hold the halves of ap, bp, cb, cs
      const uint32_t lo_next = __shfl_down(lo, 1, 64);
      if (lane >= 5 && lane <= 11 && ((lane - 5) & 1) == 0) {
        const double v = __longlong_as_double(static_cast<long long>(
            (static_cast<uint64_t>(lo_next) << 32) | lo));
        const int k = (lane - 5) >> 1;
        if (k == 0) ws.d_ap = v;
        else if (k == 1) ws.d_bp = v;
        else if (k == 2) ws.d_cb = v;
        else ws.d_cs = v;
      }
      return;
    }
    if ((it & 15) == 15 || P.spin_limit == 0) {
      uint32_t ab = 0;
      if (lane == 0) ab = ld_rlx(ws_abort(P));
      if (__shfl(ab, 0, 64) || wall_clock64() - t0 >= P.spin_limit) {
        if (lane == 0) {
          st_rlx(ws_abort(P), 1u);
          ws.help_state = 2;
        }
        return;
      }
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// Contributor c of group g until the group has no tree left (all threads).
// Returns false if the launch was abandoned.
template <typename T, class A, bool kShort>
__device__ __forceinline__ bool help_group(Lds<WgScratch>& ws, const Params& P, const A& ar, int g,
                                           int c) {
  const int tid = threadIdx.x;
  uint32_t last = 0;
  for (;;) {
    if (tid < 64) await_desc(ws, P, g, last);
    __syncthreads();
    const int state = ws.help_state;
    if (state != 0) return state == 1;
    const uint32_t seq = ws.d_seq;
    const int bn = ws.d_bn, geff = ws.d_geff, tree = ws.d_tree;
    last = seq;
    if (c < geff) {
      const TermParams tp{ws.d_cb, ws.d_cs, ws.d_ap, ws.d_bp};
      for (int p = 0; p < bn; ++p) {
        const int node = ws.d_node[p];
        const T* rb = row_ptr<T>(P, P.target, tree, node);
        const T* rs = row_ptr<T>(P, P.draft, tree, node);
        const Geom geo = row_geom(rb, P.vocab);
        const StripeResult part = stripe_pass<T, A, kShort>(ws, rb, rs, geo, stripe(geo, c, geff),
                                                    ws.d_cmd[p], tp, ar);
        if (tid == 0) {
          ws.res[p].s0 = part.s0;
          ws.res[p].s1 = part.s1;
          ws.res[p].m0 = part.m0;
          ws.res[p].m1 = part.m1;
        }
      }
      if (tid == 0) write_parts(P, ws, g, seq, bn, c, 0);
    }
    __syncthreads();
  }
}

// A workgroup whose group is done (all threads): helps a running group with
// the fewest helpers that still takes one, until none does. Workgroups that
// look at the same time spread over the groups with that fewest count: each
// starts its search at its own position.
template <typename T, class A, bool kShort>
__device__ __forceinline__ void help_others(Lds<WgScratch>& ws, const Params& P, A ar,
                                            int g_self) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int cap = P.Gx - P.G;
  const int ng = P.ngroups;
  const uint32_t start = (static_cast<uint32_t>(blockIdx.x) * 2654435761u) % static_cast<uint32_t>(ng);
  for (;;) {
    if (tid < 64) {
      // fewest helpers among the running groups that take one
      uint32_t fewest = ~0u;
      for (int gg = lane; gg < ng; gg += 64) {
        if (gg == g_self) continue;
        const uint64_t w0 = ld_rlx(&ws_desc(P, gg)[0]);
        if (static_cast<uint32_t>(w0) & kDescDone) continue;
        const uint32_t n = ld_rlx(ws_hcount(P, gg));
        if (static_cast<int>(n) < cap && n < fewest) fewest = n;
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const uint32_t o = __shfl_xor(fewest, off, 64);
        fewest = o < fewest ? o : fewest;
      }
      // the first such group from this workgroup's starting position
      uint32_t best = ~0u;    // distance from the start
      if (fewest != ~0u) {
        for (int j = lane; j < ng; j += 64) {
          const int gg = static_cast<int>((start + static_cast<uint32_t>(j)) % static_cast<uint32_t>(ng));
          if (gg == g_self) continue;
          const uint64_t w0 = ld_rlx(&ws_desc(P, gg)[0]);
          if (static_cast<uint32_t>(w0) & kDescDone) continue;
          if (ld_rlx(ws_hcount(P, gg)) == fewest) {
            best = static_cast<uint32_t>(j);
            break;
          }
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const uint32_t o = __shfl_xor(best, off, 64);
        best = o < best ? o : best;
      }
      if (lane == 0) {
        int g2 = best == ~0u ? -1 : static_cast<int>((start + best) % static_cast<uint32_t>(ng));
        int h = 0;
        if (g2 >= 0) {
          h = static_cast<int>(__hip_atomic_fetch_add(ws_hcount(P, g2), 1u, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT));
          if (h >= cap) h = -1;          // taken meanwhile: look again
        }
        ws.help_g = g2;
        ws.help_h = h;
      }
    }
    __syncthreads();
    const int g2 = ws.help_g, h = ws.help_h;
    __syncthreads();
    if (g2 < 0) return;                  // no group takes a helper
    if (h < 0) continue;
    if (!help_group<T, A, kShort>(ws, P, ar, g2, P.G + h)) return;
  }
}

// This member's share of the batch in sm.b* (all threads): its stripe of every
// pass, left in LDS. The next controller step publishes them as tagged
// partials and awaits the other contributors'.
template <typename T, class A, int kCap>
__device__ __forceinline__ void run_batch(Lds<TreeSmem<kCap>>& sm, Lds<WgScratch>& ws,
                                          const Params& P, const A& ar, int g, int m) {
  const int tid = threadIdx.x;
  const int bn = sm.bn;
  const uint32_t seq = sm.seq + 1u;
  const int b = sm.tree;
  const int geff = sm.geff;
  // Member 0 reads the group's helper count here and uses it only after the
  // stripes: the load completes under the stripes' own loads instead of
  // delaying them by a round trip.
  uint32_t hcount = 0;
  if (m == 0 && tid == 0) {
    if (geff > P.G) publish_batch(P, g, seq, sm, geff);
    hcount = ld_rlx(ws_hcount(P, g));
  }
  const TermParams tp{sm.cmd_cb, sm.cmd_cs, sm.cmd_ap, sm.cmd_bp};
  for (int p = 0; p < bn; ++p) {
    const int node = sm.bnode[p];
    const T* rb = row_ptr<T>(P, P.target, b, node);
    const T* rs = row_ptr<T>(P, P.draft, b, node);
    const Geom geo = row_geom(rb, P.vocab);
    const StripeResult part = stripe_pass<T, A, (kCap > kCapSmall)>(
        ws, rb, rs, geo, stripe(geo, m, geff), sm.bcmd[p], tp, ar);
    if (tid == 0) {
      ws.res[p].s0 = part.s0;
      ws.res[p].s1 = part.s1;
      ws.res[p].m0 = part.m0;
      ws.res[p].m1 = part.m1;
    }
  }
  if (tid == 0) {
    const int cap = P.Gx - P.G;
    const int n = static_cast<int>(hcount);
    ws.res_count = m == 0 ? static_cast<uint64_t>(n < cap ? n : cap) : 0;
    // the partials are written by the next controller step
    sm.seq = seq;
    sm.pending = 1;
    // the weights of pass 0 stay available for drawing Y at its node
    const int cmd0 = sm.bcmd[0];
    sm.spass_node = (cmd0 == kCmdSPass || cmd0 == kCmdSPassSd) ? sm.bnode[0] : -1;
    sm.last_ap = sm.cmd_ap;
    sm.last_bp = sm.cmd_bp;
    sm.last_cb = sm.cmd_cb;
    sm.last_cs = sm.cmd_cs;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------

// Clears the abort flag and the partials (tag 0: no batch yet) and gives
// every tree the outputs of an aborted tree (status TV_TREE_ABORTED, -1
// sentinels, counters 0), which finish_tree overwrites for the trees it
// finishes. Every loop is grid-stride, so any grid covers any batch.
__global__ void __launch_bounds__(256) init_kernel(Params P) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  if (i == 0) *ws_abort(P) = 0u;
  uint64_t* parts = reinterpret_cast<uint64_t*>(P.ws + P.off_parts);
  for (size_t k = i; k < P.parts_words; k += stride) parts[k] = 0u;
  uint64_t* desc = reinterpret_cast<uint64_t*>(P.ws + P.off_desc);
  for (size_t k = i; k < P.desc_words; k += stride) desc[k] = 0u;
  const size_t nb = static_cast<size_t>(P.batch);
  for (size_t b = i; b < nb; b += stride) {
    P.status[b] = TV_TREE_ABORTED;
    P.accept_len[b] = -1;
    P.accepted_node[b] = -1;
    P.bonus_token[b] = -1;
    if (P.counters) {
#pragma unroll
      for (int c = 0; c < TV_NUM_COUNTERS; ++c) P.counters[b * TV_NUM_COUNTERS + c] = 0;
    }
  }
  if (P.node_state || P.node_theta || P.p_init) {
    const size_t nn = nb * static_cast<size_t>(P.num_nodes);
    for (size_t k = i; k < nn; k += stride) {
      if (P.node_state) P.node_state[k] = TV_NODE_UNTESTED;
      if (P.node_theta) P.node_theta[k] = -1.0f;
      if (P.p_init) P.p_init[k] = -1.0f;
    }
  }
}

template <typename T, class A, int kCap>
__global__ void __launch_bounds__(kNT) verify_kernel(Params P, A ar) {
  __shared__ TreeSmem<kCap> sm_;
  __shared__ WgScratch ws_;
  __shared__ Params Ps_;     // for the controller, which is not inlined
  Lds<TreeSmem<kCap>>& sm = lds_ref(sm_);
  Lds<WgScratch>& ws = lds_ref(ws_);
  Lds<Params>& Ps = lds_ref(Ps_);
  const int tid = threadIdx.x;
  const int g = static_cast<int>(blockIdx.x) / P.G;
  const int m = static_cast<int>(blockIdx.x) - g * P.G;
  if (tid == 0) {
    Ps_ = P;
    sm.seq = 0;
    sm.geff = sm.geff_last = P.G;
    ws.stop = 0;
  }
  __syncthreads();
  bool live = true;
  for (int b = g; b < P.batch; b += P.ngroups) {
    begin_tree<T>(sm, ws, Ps, ar, b);
    for (;;) {
      controller_step<T, A>(sm, ws, Ps, ar, g, m, false);
      while (sm.cmd == kCmdLocalSample) {
        if (m == 0) local_sample<T, A>(sm, ws, Ps, ar, g);
        else if (tid == 0) sm.res_y = 0;   // Y is reported by member 0
        __syncthreads();
        controller_step<T, A>(sm, ws, Ps, ar, g, m, true);
      }
      if (sm.cmd == kCmdDone) break;
      if (sm.cmd == kCmdAbandon) {
        live = false;
        break;
      }
      run_batch<T, A>(sm, ws, P, ar, g, m);
    }
    if (!live) break;
    if (m == 0) finish_tree(sm, Ps);
  }
  if (!live) return;
  if (m == 0 && tid == 0) publish_done(P, g, sm.seq + 1u);
  // no store in flight on the way into the helpers' stripes, which then wait
  // for their loads one by one rather than for all at once
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  // the group has no tree left: help the groups that still run
  if (P.Gx > P.G) help_others<T, A, (kCap > kCapSmall)>(ws, P, ar, g);
}

// Vocabularies below this use the precise element path whatever the dtype:
// with few elements the per-element rounding of the fast path does not average.
constexpr int kPreciseBelowVocab = 16384;

// Milliseconds a wait inside the verifier may last before the launch is
// abandoned: 4000, or the value of the environment variable TV_WAIT_LIMIT_MS
// (a decimal integer in [0, 60000]; 0 abandons a launch at the first wait
// that is not satisfied at once, which tests of the abandon path use).
long long wait_limit_ms() {
  long long ms = 4000;
  if (const char* e = getenv("TV_WAIT_LIMIT_MS")) {
    char* end = nullptr;
    const long v = strtol(e, &end, 10);
    if (end != e && *end == '\0' && v >= 0 && v <= 60000) ms = v;
  }
  return ms;
}

template <typename T, class A, int kCap>
int launch_typed(Params P, A ar, hipStream_t stream) {
  // device properties and the kernel's occupancy, queried once per device
  struct DevInfo {
    int cus, clock_khz, per_cu;
  };
  constexpr int kMaxDevices = 64;
  static DevInfo info[kMaxDevices];
  static bool have[kMaxDevices];
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return TV_ERR_HIP;
  DevInfo di{};
  {
    std::lock_guard<std::mutex> lock(mu);
    if (dev < kMaxDevices && have[dev]) {
      di = info[dev];
    } else {
      if (hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev) !=
              hipSuccess ||
          hipDeviceGetAttribute(&di.clock_khz, hipDeviceAttributeWallClockRate, dev) !=
              hipSuccess ||
          hipOccupancyMaxActiveBlocksPerMultiprocessor(&di.per_cu, verify_kernel<T, A, kCap>, kNT,
                                                       0) != hipSuccess)
        return TV_ERR_HIP;
      if (dev < kMaxDevices) {
        info[dev] = di;
        have[dev] = true;
      }
    }
  }
  const int cus = di.cus, clock_khz = di.clock_khz;
  int per_cu = di.per_cu;
  if (per_cu < 1) per_cu = 1;
  long long resident = static_cast<long long>(per_cu) * (cus > 0 ? cus : 1);
  if (resident > tv::kMaxGrid) resident = tv::kMaxGrid;
  // group size: fill the device, at most kMaxGroup members and no stripe
  // narrower than 512 vectors
  const long long nvec = static_cast<long long>(P.vocab) * static_cast<long long>(sizeof(T)) / 16;
  long long G = resident / P.batch;
  if (G > kMaxGroup) G = kMaxGroup;
  if (G > nvec / 512) G = nvec / 512;
  if (G < 1) G = 1;
  long long ngroups = resident / G;
  if (ngroups > P.batch) ngroups = P.batch;
  P.G = static_cast<int>(G);
  P.ngroups = static_cast<int>(ngroups);
  // contributors a group's pass may have once helpers join: bounded so that
  // groups times contributors stay within the partials' kMaxGrid slots
  long long gmax = nvec / 512 < kMaxGroup ? nvec / 512 : kMaxGroup;
  long long gx = tv::kMaxGrid / ngroups;
  if (gx > gmax) gx = gmax;
  if (gx < G) gx = G;
  P.Gx = static_cast<int>(gx);
  P.spin_limit = static_cast<long long>(clock_khz) * wait_limit_ms();
  long long init_n = static_cast<long long>(P.parts_words);
  if (init_n < P.batch) init_n = P.batch;
  long long init_blocks = (init_n + 255) / 256;
  if (init_blocks > 1024) init_blocks = 1024;     // every loop of init_kernel is grid-stride
  hipLaunchKernelGGL(init_kernel, dim3(static_cast<unsigned>(init_blocks)), dim3(256), 0, stream,
                     P);
  if (hipGetLastError() != hipSuccess) return TV_ERR_HIP;
  // cooperative: the members of a group wait for each other, so all of them
  // must be resident at once
  void* args[] = {&P, &ar};
  const hipError_t e = hipLaunchCooperativeKernel(
      reinterpret_cast<const void*>(verify_kernel<T, A, kCap>),
      dim3(static_cast<unsigned>(ngroups * G)), dim3(kNT), args, 0, stream);
  return e == hipSuccess ? TV_OK : TV_ERR_HIP;
}

template <typename T, int kCap>
int launch_cap(const Params& P, bool precise, hipStream_t stream) {
  if constexpr (sizeof(T) == 2) {
    if (!precise) return launch_typed<T, FastArith, kCap>(P, FastArith{P.k32}, stream);
  }
  return launch_typed<T, PreciseArith, kCap>(P, PreciseArith{P.k64}, stream);
}

// ---------------------------------------------------------------------------
// Draft-tree token sampler (Def. de_tree, Sec. 3.3): the children of every
// node take tokens drawn from the node's tempered draft distribution, in
// ascending node index, each by inverse CDF (ascending token order) at its own
// uniform; without replacement, each drawn token is removed before the next
// sibling's draw. One workgroup per (tree, node) row.
// ---------------------------------------------------------------------------

struct SampleParams {
  const int32_t* parents;
  const void* draft;
  const float* uniforms;
  int32_t* tokens;
  int32_t* status;
  int batch, num_nodes, vocab, mode;
};

// chunk sums held per row: chunks of 8 units up to 16384 units (about 2^17
// bf16 tokens), larger chunks (at most 64 units) up to the vocabulary limits
// (2^17 vectors plus 14 head and tail elements)
constexpr int kSampleMaxChunks = 2056;

// The sampler's frames are integers: c(m) = -ceil(m k), so that a sum moves
// from one frame to another by an exact power of two. Terms stay at most 1
// and the fp32 frame is exact (an integer-valued fp32 on the fast path).
template <class A>
__device__ __forceinline__ double sample_frame(const A& ar, float m) {
  if constexpr (A::kPrecise) return -ceil(static_cast<double>(m) * ar.k);
  else return static_cast<double>(-ceilf(m * ar.k));
}

// v * 2^d for a frame difference d <= 0 (exact unless the result underflows)
__device__ __forceinline__ double frame_shift(double v, double d) {
  return ldexp(v, static_cast<int>(fmax(d, -4096.0)));
}

template <typename T>
struct SampleSmem {
  double cs[kSampleMaxChunks];     // chunk weight sums, in the row's frame once rescaled
  T cm[kSampleMaxChunks];          // chunk maxima, values of the row in its element format
  int32_t kids[TV_MAX_NODES];      // children of the row's node, ascending
  int32_t removed[TV_MAX_NODES];   // tokens drawn so far at this row (without replacement)
  int nkids, nremoved, owner, chunk, token;
  double W, run;
};

// the workgroup reductions' scratch, without the verifier's fields
struct SampleScratch {
  float red_f[2 * kNW];
  double scan_d[kNW];
};

// Every tree starts OK with the root's token -1; the rows then raise status.
__global__ void __launch_bounds__(256) sample_init_kernel(SampleParams S) {
  const int b = static_cast<int>(blockIdx.x * blockDim.x + threadIdx.x);
  if (b < S.batch) {
    S.status[b] = TV_TREE_OK;
    S.tokens[static_cast<size_t>(b) * S.num_nodes] = -1;
  }
}

// Every token of a tree whose status is an error becomes -1.
__global__ void __launch_bounds__(256) sample_finish_kernel(SampleParams S) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<size_t>(S.batch) * S.num_nodes) return;
  if (S.status[i / S.num_nodes] != TV_TREE_OK) S.tokens[i] = -1;
}

// The weights of one row are 2^(z*k + c) in a frame c, grouped in units:
// head elements (up to the first 16-byte boundary), 16-byte vectors, tail
// elements, in token order; consecutive units form chunks (8 units each up to
// about 2^17 bf16 tokens, more for larger rows). A unit's sum
// and the running sum inside it are formed in the same order, so a rescan
// reproduces the sum that chose it. Tokens already drawn (without
// replacement) weigh 0.
template <typename T, class A>
struct RowWeights {
  static constexpr int E = Elem<T>::E;
  using W = typename Terms<A, false, false>::W;
  const T* row;
  Geom g;
  A ar;
  const Lds<SampleSmem<T>>* sm;

  __device__ int units() const { return g.head + g.nvec + g.tail; }
  __device__ int first(int u) const {
    if (u < g.head) return u;
    if (u < g.head + g.nvec) return g.head + (u - g.head) * E;
    return g.head + g.nvec * E + (u - g.head - g.nvec);
  }
  __device__ int count(int u) const { return (u >= g.head && u < g.head + g.nvec) ? E : 1; }
  __device__ bool drawn(int x) const {
    for (int r = 0; r < sm->nremoved; ++r)
      if (sm->removed[r] == x) return true;
    return false;
  }
  __device__ void load(int u, float (&x)[E]) const {
    if (count(u) == E) {
      Elem<T>::unpack(load16(row, g.head, u - g.head), x);
    } else {
      x[0] = Elem<T>::scalar(row + first(u));
#pragma unroll
      for (int e = 1; e < E; ++e) x[e] = -INFINITY;
    }
  }
  __device__ float vmax(const float (&x)[E]) const {
    float m = x[0];
#pragma unroll
    for (int e = 1; e < E; ++e) m = fmaxf(m, x[e]);
    return m;
  }
  __device__ W weight(int x, float z, double c) const {
    if (sm->nremoved && drawn(x)) return W(0);
    if constexpr (A::kPrecise) return ar.ex(z, c);
    else return fast_exp2(fmaf(z, ar.k, static_cast<float>(c)));
  }
  // sum of unit u's weights in frame c, its values already loaded
  __device__ double sum_of(int u, const float (&x)[E], double c) const {
    const int n = count(u), x0 = first(u);
    W acc = W(0);
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (e < n) acc += weight(x0 + e, x[e], c);
    return static_cast<double>(acc);
  }
  __device__ double unit_sum(int u, double c) const {
    float x[E];
    load(u, x);
    return sum_of(u, x, c);
  }
  // first element of unit u whose running sum, after `run`, passes target
  // (-1 if none); the last element of positive weight goes to *lastpos
  __device__ int find(int u, double c, double run, double target, int* lastpos) const {
    float x[E];
    load(u, x);
    const int n = count(u), x0 = first(u);
    W acc = W(0);
    int found = -1;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if (e < n && found < 0) {
        const W w = weight(x0 + e, x[e], c);
        acc += w;
        if (w > W(0)) {
          *lastpos = x0 + e;
          if (run + static_cast<double>(acc) > target) found = x0 + e;
        }
      }
    }
    return found;
  }
};

template <typename T, class A>
__global__ void __launch_bounds__(kNT) sample_kernel(SampleParams S, A ar) {
  __shared__ SampleSmem<T> sm_;
  __shared__ SampleScratch ws_;
  Lds<SampleSmem<T>>& sm = lds_ref(sm_);
  Lds<SampleScratch>& ws = lds_ref(ws_);
  const int tid = threadIdx.x, lane = tid & 63;
  const int n1 = S.num_nodes;
  const int b = static_cast<int>(blockIdx.x / static_cast<unsigned>(n1));
  const int j = static_cast<int>(blockIdx.x - static_cast<unsigned>(b) * n1);
  const int32_t* par = S.parents + static_cast<size_t>(b) * n1;

  // the tree's links (every row checks them) and whether this node has
  // children: a row without children (about half of them) stops here
  int bad = 0, anykid = 0;
  for (int i = tid; i < n1; i += kNT) {
    const int p = par[i];
    if (i == 0 ? p != -1 : (p < 0 || p >= i)) bad = 1;
    if (i > 0 && p == j) anykid = 1;
  }
  if (__syncthreads_or(bad)) {
    if (j == 0 && tid == 0) atomicMax(&S.status[b], static_cast<int32_t>(TV_TREE_BAD_PARENT));
    return;
  }
  if (!__syncthreads_or(anykid)) return;
  // the children in order
  if (tid == 0) {
    sm.nkids = 0;
    sm.nremoved = 0;
  }
  __syncthreads();
  for (int base = 0; base < n1; base += kNT) {
    const int i = base + tid;
    const bool kid = i < n1 && i > 0 && par[i] == j;
    const double inc = block_incl_scan(ws, kid ? 1.0 : 0.0);
    const int before = sm.nkids;
    if (kid) sm.kids[before + static_cast<int>(inc) - 1] = i;
    __syncthreads();
    if (tid == kNT - 1) sm.nkids = before + static_cast<int>(inc);
    __syncthreads();
  }
  const int nk = sm.nkids;

  const T* row = static_cast<const T*>(S.draft) + (static_cast<size_t>(b) * n1 + j) *
                                                      static_cast<size_t>(S.vocab);
  const RowWeights<T, A> rw{row, row_geom(row, S.vocab), ar, &sm};
  constexpr int E = RowWeights<T, A>::E;
  const int U = rw.units();
  // chunks of cu consecutive units, cu a multiple of 8, at most
  // kSampleMaxChunks of them (cu = 8 up to about 2^17 bf16 tokens)
  const int cu = 8 * max(1, (U + 8 * kSampleMaxChunks - 1) / (8 * kSampleMaxChunks));
  const int C = (U + cu - 1) / cu;
  if (C > kSampleMaxChunks || cu > 64) {   // beyond the vocabulary limits the host checks
    if (tid == 0) atomicMax(&S.status[b], static_cast<int32_t>(TV_TREE_DEGENERATE));
    return;
  }

  // One read of the row. Thread t sums chunks t, t + 256, ... on its own, 8
  // units at a time (8 16-byte vectors, or head and tail elements at the two
  // ends of the row), the next 8 units' loads in flight while the current ones
  // are summed; a chunk keeps the frame of its running maximum (Online). No
  // reduction across threads until the row is read. A chunk's sum is the
  // fp64 sum of its units' sums, each of those formed as the draw's rescan
  // forms it (fp32 terms added in fp32 on the fast path, fp64 on the precise
  // one), and is moved into the row's frame by an fp64 factor.
  const int nsb = cu / 8;                        // 8-unit blocks per chunk
  const int my_chunks = C > tid ? (C - tid + kNT - 1) / kNT : 0;
  const int items = my_chunks * nsb;
  auto block_unit = [&](int i) { return (tid + kNT * (i / nsb)) * cu + 8 * (i % nsb); };
  auto pure = [&](int ub) { return ub >= rw.g.head && ub + 8 <= rw.g.head + rw.g.nvec; };
  auto load_block = [&](int ub, uint4 (&v)[8]) {
    if (pure(ub)) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = load16(row, rw.g.head, ub - rw.g.head + e);
    }
  };
  float tmax = -INFINITY;
  const Online o0{-INFINITY, sample_frame(ar, kFrameSentinel), 0.0};
  Online o = o0;
  uint4 cur[8], nxt[8];
  if (items > 0) load_block(block_unit(0), cur);
  for (int i = 0; i < items; ++i) {
    if (i + 1 < items) load_block(block_unit(i + 1), nxt);
    const int ub = block_unit(i);
    if (i % nsb == 0) o = o0;
    float vmax = -INFINITY;
    const bool pb = pure(ub);
    if (pb) {
      // the values are unpacked again for the sums rather than kept: the
      // 8 x E floats would hold registers that the loads in flight need
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pin(cur[e]);
        float t[E];
        Elem<T>::unpack(cur[e], t);
#pragma unroll
        for (int q = 0; q < E; ++q) vmax = fmaxf(vmax, t[q]);
      }
    } else {
      for (int e = 0; e < 8; ++e) {
        if (ub + e < U) {
          float t[E];
          rw.load(ub + e, t);
#pragma unroll
          for (int q = 0; q < E; ++q) vmax = fmaxf(vmax, t[q]);
        }
      }
    }
    if (vmax > o.m) {
      const double cn = sample_frame(ar, vmax);
      o.s = frame_shift(o.s, cn - o.c);
      o.m = vmax;
      o.c = cn;
    }
    // a unit's sum is formed as a rescan forms it (its terms in order, in the
    // precision of the terms), and unit sums are added in fp64
    const float cf32 = static_cast<float>(o.c);
    auto add_unit = [&](const float (&t)[E]) {
      if constexpr (A::kPrecise) {
        double acc = 0.0;
#pragma unroll
        for (int q = 0; q < E; ++q) acc += ar.ex(t[q], o.c);
        o.s += acc;
      } else {
        float acc = 0.0f;
#pragma unroll
        for (int q = 0; q < E; ++q) acc += fast_exp2(fmaf(t[q], ar.k, cf32));
        o.s += static_cast<double>(acc);
      }
    };
    if (pb) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pin(cur[e]);
        float t[E];
        Elem<T>::unpack(cur[e], t);
        add_unit(t);
      }
    } else {
      for (int e = 0; e < 8; ++e) {
        if (ub + e < U) {
          float t[E];
          rw.load(ub + e, t);
          add_unit(t);
        }
      }
    }
    if (i % nsb == nsb - 1) {
      const int c = tid + kNT * (i / nsb);
      // the sum in the frame of the chunk's maximum (that of the sentinel, with
      // sum 0 or NaN, when the chunk has no finite value); the maximum is a
      // value of the row, kept in the row's element format
      sm.cs[c] = o.s;
      sm.cm[c] = Elem<T>::narrow(o.m);
      tmax = fmaxf(tmax, o.m);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) cur[e] = nxt[e];
  }
  float rowmax = tmax, unused_max = -INFINITY;
  block_max2(ws, rowmax, unused_max);
  if (!(rowmax > -INFINITY) || rowmax == INFINITY) {
    if (tid == 0) atomicMax(&S.status[b], static_cast<int32_t>(TV_TREE_NONFINITE));
    return;
  }
  const double cf = sample_frame(ar, rowmax);   // the row's frame

  // chunk sums into the row's frame; thread t owns the chunks [cb, ce)
  const int cb = static_cast<int>(static_cast<long long>(C) * tid / kNT);
  const int ce = static_cast<int>(static_cast<long long>(C) * (tid + 1) / kNT);
  double ts = 0.0;
  int nonfinite = 0;
  for (int c = cb; c < ce; ++c) {
    const float M = Elem<T>::widen(sm.cm[c]);
    double v = sm.cs[c];
    if (M > -INFINITY) {
      v = frame_shift(v, cf - sample_frame(ar, M));
    }
    if (!isfinite(v)) nonfinite = 1;
    sm.cs[c] = v;
    ts += v;
  }
  nonfinite = __syncthreads_or(nonfinite);
  if (nonfinite) {
    if (tid == 0) atomicMax(&S.status[b], static_cast<int32_t>(TV_TREE_NONFINITE));
    return;
  }

  for (int k = 0; k < nk; ++k) {
    const int child = sm.kids[k];
    const double incl = block_incl_scan(ws, ts);
    if (tid == kNT - 1) sm.W = incl;
    if (tid == 0) sm.owner = kNT;
    __syncthreads();
    const double W = sm.W;
    if (!(W > 0.0)) {          // every token already drawn: not enough tokens for the siblings
      if (tid == 0) atomicMax(&S.status[b], static_cast<int32_t>(TV_TREE_DEGENERATE));
      return;
    }
    const double target =
        static_cast<double>(S.uniforms[static_cast<size_t>(b) * n1 + child]) * W;
    if (incl > target)
      __hip_atomic_fetch_min(&sm.owner, tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __syncthreads();
    const int owner = sm.owner;     // < kNT: the last thread's sum is W > target
    if (tid == owner) {
      // the owner's chunk holding the target (else its last chunk of positive weight)
      double run = incl - ts;
      int hit = -1, lastc = -1;
      for (int c = cb; c < ce && hit < 0; ++c) {
        if (sm.cs[c] > 0.0) lastc = c;
        if (sm.cs[c] > 0.0 && run + sm.cs[c] > target) hit = c;
        else run += sm.cs[c];
      }
      if (hit < 0) {
        hit = lastc;
        run = -INFINITY;            // take its last token of positive weight
      }
      sm.chunk = hit;
      sm.run = run;
    }
    __syncthreads();
    if (tid < 64) {
      // wave 0 rescans the chunk, one unit per lane, in the row's frame
      const int c = sm.chunk;
      int tok = -1;
      if (c >= 0) {
        const int u = c * cu + lane;
        const bool mine = lane < cu && u < U;
        const double us = mine ? rw.unit_sum(u, cf) : 0.0;
        double inc = us;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const double o = __shfl_up(inc, off, 64);
          if (lane >= off) inc += o;
        }
        const double run = sm.run;
        const uint64_t pos = __ballot(us > 0.0);
        const uint64_t hitm = __ballot(mine && us > 0.0 && run + inc > target);
        const int L = hitm ? __ffsll(static_cast<unsigned long long>(hitm)) - 1
                           : (pos ? 63 - __clzll(static_cast<long long>(pos)) : -1);
        int t = -1, lp = -1;
        if (L >= 0 && lane == L) {
          t = rw.find(u, cf, hitm ? run + (inc - us) : -INFINITY, target, &lp);
          if (t < 0) t = lp;        // rounding left the boundary just short of the unit's end
        }
        if (L >= 0) tok = __shfl(t, L, 64);
      }
      if (lane == 0) {
        sm.token = tok;
        S.tokens[static_cast<size_t>(b) * n1 + child] = tok;
        if (tok < 0) atomicMax(&S.status[b], static_cast<int32_t>(TV_TREE_DEGENERATE));
      }
    }
    __syncthreads();
    const int tok = sm.token;
    if (tok < 0) return;
    if (S.mode == TV_SIBLINGS_WITHOUT_REPLACEMENT && k + 1 < nk) {
      // the token leaves its chunk's sum and the owning thread's
      const int u = tok < rw.g.head ? tok
                    : (tok < rw.g.head + rw.g.nvec * RowWeights<T, A>::E
                           ? rw.g.head + (tok - rw.g.head) / RowWeights<T, A>::E
                           : rw.g.head + rw.g.nvec + (tok - rw.g.head - rw.g.nvec * RowWeights<T, A>::E));
      const int c = u / cu;
      if (tid == 0) sm.removed[sm.nremoved++] = tok;
      __syncthreads();
      // The chunk's sum is formed again from its units, the drawn token now
      // weighing 0. Subtracting the token's weight instead would cancel: when
      // it held most of the row's mass, the rounding of the old sum (relative
      // to the old total) would be large against the new total.
      if (tid < 64) {
        const int uu = c * cu + lane;
        const double us = (lane < cu && uu < U) ? rw.unit_sum(uu, cf) : 0.0;
        const double v = wave_sum(us);
        if (lane == 0) sm.cs[c] = v;
      }
      __syncthreads();
      if (c >= cb && c < ce) {
        ts = 0.0;
        for (int cc = cb; cc < ce; ++cc) ts += sm.cs[cc];
      }
      __syncthreads();
    }
  }
}

template <typename T, class A>
int launch_sample_typed(const SampleParams& S, A ar, hipStream_t stream) {
  const long long rows = static_cast<long long>(S.batch) * S.num_nodes;
  hipLaunchKernelGGL(sample_init_kernel, dim3(static_cast<unsigned>((S.batch + 255) / 256)),
                     dim3(256), 0, stream, S);
  if (hipGetLastError() != hipSuccess) return TV_ERR_HIP;
  hipLaunchKernelGGL((sample_kernel<T, A>), dim3(static_cast<unsigned>(rows)), dim3(kNT), 0,
                     stream, S, ar);
  if (hipGetLastError() != hipSuccess) return TV_ERR_HIP;
  hipLaunchKernelGGL(sample_finish_kernel, dim3(static_cast<unsigned>((rows + 255) / 256)),
                     dim3(256), 0, stream, S);
  return hipGetLastError() == hipSuccess ? TV_OK : TV_ERR_HIP;
}

}  // namespace

namespace tv {

int launch(const VerifyArgs& a, Algo algo, void* workspace, hipStream_t stream) {
  const WorkspaceLayout L = workspace_layout(a.batch, a.vocab);
  Params P{};
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
  P.tmax = a.target_max;
  P.tsum = a.target_sum;
  P.dmax = a.draft_max;
  P.dsum = a.draft_sum;
  P.ws = static_cast<uint8_t*>(workspace);
  P.off_parts = L.off_parts;
  P.parts_words = L.parts_bytes / 8;
  P.off_desc = L.off_desc;
  P.desc_words = L.desc_bytes / 8;
  P.batch = a.batch;
  P.num_nodes = a.num_nodes;
  P.vocab = a.vocab;
  P.mode = a.mode;
  P.algo = static_cast<int>(algo);
  P.early = a.node_theta == nullptr ? 1 : 0;
  P.k64 = 1.4426950408889634 / static_cast<double>(a.temperature);
  P.k32 = static_cast<float>(P.k64);
  const bool precise = a.dtype == TV_DTYPE_F32 || a.vocab < kPreciseBelowVocab;
  const bool small = a.num_nodes <= kCapSmall;
  if (a.dtype == TV_DTYPE_BF16)
    return small ? launch_cap<uint16_t, kCapSmall>(P, precise, stream)
                 : launch_cap<uint16_t, kCapLarge>(P, precise, stream);
  return small ? launch_cap<float, kCapSmall>(P, true, stream)
               : launch_cap<float, kCapLarge>(P, true, stream);
}

}  // namespace tv

// Device scratch of tv_verify_noalloc: the workspace of its calls, one copy on
// every device the library runs on, held until the process ends. Host code
// never uses this name as a device address: static_scratch looks up each
// device's address once and every launch passes that address.
static __device__ __align__(256) uint8_t scratch[tv::kStaticScratchBytes];

namespace tv {

int static_scratch(void** ptr, size_t* bytes) {
  constexpr int kMaxDevices = 64;
  static void* addr[kMaxDevices];
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TV_ERR_HIP;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TV_ERR_HIP;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = kStaticScratchBytes;
  return TV_OK;
}

int launch_sample(const SampleArgs& a, hipStream_t stream) {
  SampleParams S{a.parents, a.draft, a.uniforms, a.tokens, a.status,
                 a.batch, a.num_nodes, a.vocab, a.mode};
  const double k64 = 1.4426950408889634 / static_cast<double>(a.temperature);
  const bool precise = a.dtype == TV_DTYPE_F32 || a.vocab < kPreciseBelowVocab;
  if (a.dtype == TV_DTYPE_BF16) {
    if (!precise) return launch_sample_typed<uint16_t>(S, FastArith{static_cast<float>(k64)}, stream);
    return launch_sample_typed<uint16_t>(S, PreciseArith{k64}, stream);
  }
  return launch_sample_typed<float>(S, PreciseArith{k64}, stream);
}

}  // namespace tv
