// LM head with fused row statistics for gfx950: logits = hidden * weight^T on
// bf16 MFMA, rounded to bf16, and in the same kernel the statistics of every
// row of the rounded logits that the verifier's tempered softmax needs (the
// row maximum and the sum of exp((z - max) / T)), so that no pass over the
// logits is needed to compute them (the distributions M_b and M_s of the
// problem statement, Alg. 3 REQUIRE, are softmax(logits / T) per row).
//
// Tiling. A workgroup of 256 threads (4 wavefronts, 2 x 2) computes a 256 x 256
// tile of logits; each wavefront a 128 x 128 sub-tile as 4 x 4 blocks of
// v_mfma_f32_32x32x16_bf16 (fp32 accumulation, 256 accumulator registers per
// lane, one wavefront per SIMD). K advances 64 at a time through two LDS
// buffers: while the products of one K-slice are formed from one buffer, the
// slice after next of both operand tiles is loaded from global memory into
// registers (16-byte loads, coalesced along K) and the next one is stored
// into the other buffer, so one barrier per K-slice suffices; the loads and
// stores are spread evenly over the products. Both operands are K-contiguous
// (hidden [M][K], weight [N][K]), so every MFMA operand fragment is one
// 16-byte LDS read; LDS rows are padded by 16 bytes against bank conflicts.
// Each XCD gets a contiguous run of tiles, ordered in bands of 8 row tiles
// column tile by column tile, so the tiles it runs at once read each slice of
// the hidden states and of the weight once from HBM and share it through the
// XCD's L2.
//
// Epilogue. Each accumulator is rounded to bf16 (round to nearest even, by the
// hardware conversion) into the tile in LDS; the tile is stored in 16-byte
// vectors along its rows; then each thread reads one row of it back and forms
// the row's maximum and its sum of 2^((z - max) k), k = log2(e)/T, in fp32:
// one (max, sum) partial per row and column tile. A second kernel merges a
// row's partials in fp64, each moved to the frame of the row maximum.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tv.h"
#include "tv_launch.h"

namespace {

constexpr int kBM = 256, kBN = tv::kLmheadTileN, kBK = 64;
constexpr int kLds = kBK + 8;          // padded LDS row, bf16 elements (144 bytes)
constexpr int kThreads = 256;
constexpr int kGroupM = 8;             // row tiles per band of the tile order
constexpr int kVecs = kBM * kBK / 8 / kThreads;   // 16-byte vectors per thread and operand
static_assert(kBM == kBN, "one load pattern serves both operands");

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

struct LmParams {
  const uint16_t* x;      // [M][K] bf16 bits
  const uint16_t* w;      // [N][K] bf16 bits
  uint16_t* logits;       // [M][N] bf16 bits
  float* part_max;        // [M][tiles_n]
  float* part_sum;        // [M][tiles_n], in the frame of part_max
  float* row_max;         // [M]
  double* row_sum;        // [M]
  int M, K, N, tiles_n;
  float k32;              // log2(e) / T rounded to fp32
};

// One K-slice of a 256-row operand tile: 2048 16-byte vectors, eight per
// thread (vector v = thread + 256 q: row v / 8, 8 bf16 at column 8 (v % 8)).
// The loads are buffer loads over the tile's rows: the hardware returns zeros
// for a vector beyond the last row of the matrix, and a vector beyond the
// last column is given an offset past the range (at most 256 rows of 2^16
// bf16, 32 MiB), so no load branches.
constexpr int kBufferConfig = 0x00020000;   // buffer descriptor word 3 on gfx9-family GPUs

struct Slice {
  uint4 v[kVecs];
  __device__ __forceinline__ static __amdgpu_buffer_rsrc_t tile(const uint16_t* base, int rows,
                                                                int row0, int K) {
    const int nrows = min(kBM, rows - row0);
    return __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(base + static_cast<size_t>(row0) * K), 0,
        nrows * K * static_cast<int>(sizeof(uint16_t)), kBufferConfig);
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, int K, int k0) {
#pragma unroll
    for (int q = 0; q < kVecs; ++q) {
      const int idx = threadIdx.x + kThreads * q;
      const int c = k0 + 8 * (idx & 7);
      const int past = (K - 1 - c) >> 31;      // -1 beyond the last column, else 0
      const int off = (((idx >> 3) * K + c) * static_cast<int>(sizeof(uint16_t))) |
                      (past & 0x7fffffff);      // at least 2^31 - 1 > range: reads zeros
      v[q] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
    }
  }
  __device__ __forceinline__ void store(uint16_t* lds) const {
#pragma unroll
    for (int q = 0; q < kVecs; ++q) {
      const int idx = threadIdx.x + kThreads * q;
      *reinterpret_cast<uint4*>(lds + (idx >> 3) * kLds + 8 * (idx & 7)) = v[q];
    }
  }
};

__device__ __forceinline__ bf16x8 frag(const uint16_t* lds, int off) {
  const uint4 u = *reinterpret_cast<const uint4*>(lds + off);
  return __builtin_bit_cast(bf16x8, u);
}

constexpr int kOperandLds = kBM * kLds;       // bf16 elements of one operand buffer
constexpr int kTilePitch = kBN + 8;           // bf16 elements per row of the rounded tile in LDS
static_assert((kBM / 2) * kTilePitch <= 2 * kOperandLds, "half the rounded tile fits a buffer");

// Statistics of one row of the rounded tile in LDS over its first `cols`
// columns (kCols > 0: all kCols, with no masking), in one pass: the running
// maximum m and the sum of 2^(z k + c) in the frame c = -m k (fp32 product);
// when a group of 8 values raises the maximum, the partial sums move to the
// new frame by 2^(c_new - c_old). At the end the frame is that of the row's
// maximum, as if the terms had been formed with it. The hardware exp2 gives 0
// for -inf, so a row whose columns are all -inf sums 0 (its frame never
// moves); NaN or +inf propagate into the sum (NaN is not ordered by fmaxf and
// surfaces there; +inf makes the frame -inf and its term NaN).
template <int kCols>
__device__ __forceinline__ void row_stats(const uint16_t* tr, int cols, float k, float& m_out,
                                          float& s_out) {
  float m = -INFINITY, c = 0.0f;
  float sm[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
  for (int j = 0; j < kBN / 8; ++j) {
    const uint4 q = *reinterpret_cast<const uint4*>(tr + 8 * j);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
    float z[8];
    float gm = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      z[e] = __uint_as_float(e & 1 ? w[e >> 1] & 0xffff0000u : w[e >> 1] << 16);
      if (kCols == 0 && 8 * j + e >= cols) z[e] = -INFINITY;
      gm = fmaxf(gm, z[e]);
    }
    if (gm > m) {
      const float cn = -gm * k;
      const float f = m > -INFINITY ? __builtin_amdgcn_exp2f(cn - c) : 1.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) sm[i] *= f;
      m = gm;
      c = cn;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) sm[e & 3] += __builtin_amdgcn_exp2f(fmaf(z[e], k, c));
  }
  m_out = m;
  s_out = (sm[0] + sm[1]) + (sm[2] + sm[3]);
}

__global__ void __launch_bounds__(kThreads) lmhead_kernel(LmParams P) {
  // two buffers of both operand slices, separate arrays so that stores into
  // one can be scheduled among the reads of the other; after the products,
  // rows 0-127 of the rounded tile go into the first, rows 128-255 into the
  // second
  __shared__ __attribute__((aligned(16))) uint16_t lds0[2 * kOperandLds];
  __shared__ __attribute__((aligned(16))) uint16_t lds1[2 * kOperandLds];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  // Workgroups are dealt to the 8 XCDs in turn (workgroup i to XCD i % 8):
  // the remap gives each XCD a contiguous run of logical tiles (any grid
  // size), and the logical order walks bands of kGroupM row tiles column tile
  // by column tile, so the tiles an XCD runs at once share each operand slice
  // through its L2.
  const unsigned nb = gridDim.x, per = nb / 8u, rem = nb % 8u;
  const unsigned xcd = blockIdx.x % 8u, idx = blockIdx.x / 8u;
  const unsigned lb = xcd < rem ? xcd * (per + 1u) + idx : rem * (per + 1u) + (xcd - rem) * per + idx;
  const int tiles_m = (P.M + kBM - 1) / kBM;
  const int band = static_cast<int>(lb) / (kGroupM * P.tiles_n);
  const int in_band = static_cast<int>(lb) - band * kGroupM * P.tiles_n;
  const int gm = min(kGroupM, tiles_m - band * kGroupM);
  const int tm = band * kGroupM + in_band % gm;
  const int tn = in_band / gm;
  const int m0 = tm * kBM, n0 = tn * kBN;

  f32x16 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

  const __amdgpu_buffer_rsrc_t ra = Slice::tile(P.x, P.M, m0, P.K);
  const __amdgpu_buffer_rsrc_t rb = Slice::tile(P.w, P.N, n0, P.K);
  const int lr = lane & 31, lh = lane >> 5;
  const int nk = (P.K + kBK - 1) / kBK;
  const int fra = (wm * 128 + lr) * kLds + 8 * lh;      // this lane's fragment offsets
  const int frb = (wn * 128 + lr) * kLds + 8 * lh;
  // Two register sets of slices: slice kt + 1 waits in one while slice
  // kt + 2 is loaded into the other.
  Slice sa[2], sb[2];
  sa[0].load(ra, P.K, 0);
  sb[0].load(rb, P.K, 0);
  sa[0].store(lds0);
  sb[0].store(lds0 + kOperandLds);
  sa[1].load(ra, P.K, kBK);
  sb[1].load(rb, P.K, kBK);
  __syncthreads();
  // One K-slice: the products of slice kt from LDS buffer kt % 2 while slice
  // kt + 2 is loaded into a register set (beyond the last slice every
  // vector is past the range and reads zeros) and slice kt + 1 is stored from
  // its set into the other buffer, which was last read before the previous
  // barrier (after the last slice it is stored into the buffer no one reads
  // again). The barrier comes after the third of the four 16-deep steps, so
  // the first fragments of slice kt + 1 are read during the fourth.
  // Fragments: A single buffered (reloaded as soon as the four products that
  // read it are issued), B double buffered. The first fragments of slice 0:
  bf16x8 fa[4], fb[2][4];
#pragma unroll
  for (int a = 0; a < 4; ++a) fa[a] = frag(lds0, fra + a * 32 * kLds);
#pragma unroll
  for (int b = 0; b < 4; ++b) fb[0][b] = frag(lds0 + kOperandLds, frb + b * 32 * kLds);
  auto slice = [&](const int kt, const uint16_t* As, uint16_t* nxt, Slice& la, Slice& lb,
                   const Slice& ka, const Slice& kb) {
    // la/lb receive slice kt + 2; ka/kb hold slice kt + 1
    const uint16_t* Bs = As + kOperandLds;
    la.load(ra, P.K, (kt + 2) * kBK);
    lb.load(rb, P.K, (kt + 2) * kBK);
    // steps 0-2: products, with the fragments of the next step read from this
    // slice's buffer and slice kt + 1 stored into the other buffer
#pragma unroll
    for (int s = 0; s < kBK / 16 - 1; ++s) {
      const int cur = s & 1;
#pragma unroll
      for (int a = 0; a < 4; ++a) {
#pragma unroll
        for (int b = 0; b < 4; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[cur][b], acc[a][b],
                                                              0, 0, 0);
        fa[a] = frag(As, fra + a * 32 * kLds + 16 * (s + 1));
        fb[cur ^ 1][a] = frag(Bs, frb + a * 32 * kLds + 16 * (s + 1));
      }
    }
    ka.store(nxt);
    kb.store(nxt + kOperandLds);
    // instruction order before the barrier: rounds of (a product, a global
    // load, a product, an LDS store of the next slice, a product, two
    // fragment reads), so the loads and the stores spread over the products
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (i < 12) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    // Every wave has stored its part of slice kt + 1 and read the last
    // fragments it needs from this slice's buffer: after the barrier, the
    // other buffer holds slice kt + 1, and this one may be overwritten (by
    // the stores of slice kt + 2, during the next slice's steps 0-2).
    __syncthreads();
    // step 3: the last products of this slice, with the first fragments of
    // slice kt + 1 read from the other buffer meanwhile
    {
      constexpr int s = kBK / 16 - 1;
      constexpr int cur = s & 1;
      static_assert(cur == 1, "step 3 hands fa and fb[0] to the next slice");
#pragma unroll
      for (int a = 0; a < 4; ++a) {
#pragma unroll
        for (int b = 0; b < 4; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[cur][b], acc[a][b],
                                                              0, 0, 0);
        fa[a] = frag(nxt, fra + a * 32 * kLds);
        fb[cur ^ 1][a] = frag(nxt + kOperandLds, frb + a * 32 * kLds);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
    }
  };
  // an odd count of slices gets one more, of zeros (every vector of it is
  // past the range), which adds nothing to the products
  for (int kt = 0; kt < nk; kt += 2) {
    slice(kt, lds0, lds1, sa[0], sb[0], sa[1], sb[1]);
    slice(kt + 1, lds1, lds0, sa[1], sb[1], sa[0], sb[0]);
  }
  __syncthreads();   // the last fragment reads are done before the tile overwrites the buffers

  // Epilogue. Accumulator r of block (a, b) holds row
  // 128 wm + 32 a + 8 (r / 4) + 4 lh + r % 4 and column 128 wn + 32 b + lr of
  // the tile. The rounded tile goes through LDS (the operand buffers are free
  // now): stored from there in 16-byte vectors along rows, and read back one
  // row per thread for the statistics, so no value crosses lanes.
  // tile row R lives in row R % 128 of the first (R < 128) or second array
  auto tile_row = [&](int row) -> uint16_t* {
    return (row < kBM / 2 ? lds0 : lds1) + (row & (kBM / 2 - 1)) * kTilePitch;
  };
  uint16_t* mine = wm == 0 ? lds0 : lds1;                 // this wavefront's 128 rows
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int col = wn * 128 + b * 32 + lr;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        // the hardware conversion (v_cvt_pk_bf16_f32) rounds to nearest even
        mine[row * kTilePitch + col] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(acc[a][b][r]));
      }
    }
  __syncthreads();
  // logits: thread t stores column vector t % 32 of rows t / 32, t / 32 + 8,
  // ... (a row's 32 vectors by 32 consecutive threads), non-temporal: the
  // logits are not read again by this kernel and should not displace the
  // operand slices in the caches
  const int cols = min(kBN, P.N - n0), rows = min(kBM, P.M - m0);
  uint16_t* out = P.logits + static_cast<size_t>(m0) * P.N + n0;
  if ((P.N & 7) == 0 && (reinterpret_cast<uintptr_t>(P.logits) & 15) == 0) {
    typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
    const int c8 = 8 * (tid & 31);
    if (c8 < cols) {                                      // cols is a multiple of 8 here
      uint16_t* dst = out + static_cast<size_t>(tid >> 5) * P.N + c8;
      const size_t step = static_cast<size_t>(8) * P.N;
#pragma unroll 8
      for (int row = tid >> 5; row < rows; row += 8) {
        __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(tile_row(row) + c8),
                                    reinterpret_cast<u32x4*>(dst));
        dst += step;
      }
    }
  } else {
    for (int e = tid; e < kBM * kBN; e += kThreads) {
      const int row = e >> 8, c = e & 255;
      if (row < rows && c < cols) out[static_cast<size_t>(row) * P.N + c] = tile_row(row)[c];
    }
  }
  // statistics of row tid over the tile's columns
  if (tid < rows) {
    float m, sum;
    if (cols == kBN) {
      row_stats<kBN>(tile_row(tid), kBN, P.k32, m, sum);
    } else {
      row_stats<0>(tile_row(tid), cols, P.k32, m, sum);
    }
    const int row = m0 + tid;
    P.part_max[static_cast<size_t>(row) * P.tiles_n + tn] = m;
    P.part_sum[static_cast<size_t>(row) * P.tiles_n + tn] = sum;
  }
}

// Merges the column-tile partials of one row per wavefront (fp64 sum, each
// partial moved from its frame to the row maximum's by 2^(frame difference),
// evaluated in fp64).
__global__ void __launch_bounds__(kThreads) lmhead_merge_kernel(LmParams P) {
  const int lane = threadIdx.x & 63;
  const int row = static_cast<int>(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
  if (row >= P.M) return;
  const float* pm = P.part_max + static_cast<size_t>(row) * P.tiles_n;
  const float* ps = P.part_sum + static_cast<size_t>(row) * P.tiles_n;
  float m = -INFINITY;
  for (int t = lane; t < P.tiles_n; t += 64) m = fmaxf(m, pm[t]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  // each partial is in the frame -max_t * k (an fp32 product): move it to the
  // row's frame -m * k by 2 to the difference of the two frames
  const double cm = static_cast<double>(-m * P.k32);
  double s = 0.0;
  for (int t = lane; t < P.tiles_n; t += 64) {
    const float mt = pm[t];
    const double st = static_cast<double>(ps[t]);
    s += (mt > -INFINITY && m > -INFINITY)
             ? st * exp2(cm - static_cast<double>(-mt * P.k32))
             : st;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) {
    // from the frame -m * k rounded to fp32 to the exact frame of the maximum,
    // so that row_sum is sum exp((z - m) / T) as defined
    P.row_max[row] = m;
    P.row_sum[row] = m > -INFINITY && isfinite(m)
                         ? s * exp2(-(cm + static_cast<double>(m) * static_cast<double>(P.k32)))
                         : s;
  }
}

}  // namespace

namespace tv {

int launch_lmhead(const LmheadArgs& a, void* workspace, hipStream_t stream) {
  const LmheadLayout L = lmhead_layout(a.rows, a.vocab);
  LmParams P{};
  P.x = static_cast<const uint16_t*>(a.hidden);
  P.w = static_cast<const uint16_t*>(a.weight);
  P.logits = static_cast<uint16_t*>(a.logits);
  P.part_max = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + L.off_max);
  P.part_sum = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + L.off_sum);
  P.row_max = a.row_max;
  P.row_sum = a.row_sum;
  P.M = a.rows;
  P.K = a.hidden_size;
  P.N = a.vocab;
  P.tiles_n = L.tiles_n;
  P.k32 = static_cast<float>(1.4426950408889634 / static_cast<double>(a.temperature));
  const long long tiles_m = (a.rows + kBM - 1) / kBM;
  const long long grid = tiles_m * L.tiles_n;
  hipLaunchKernelGGL(lmhead_kernel, dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0, stream,
                     P);
  if (hipGetLastError() != hipSuccess) return TV_ERR_HIP;
  hipLaunchKernelGGL(lmhead_merge_kernel, dim3(static_cast<unsigned>((a.rows + 3) / 4)),
                     dim3(kThreads), 0, stream, P);
  return hipGetLastError() == hipSuccess ? TV_OK : TV_ERR_HIP;
}

}  // namespace tv
