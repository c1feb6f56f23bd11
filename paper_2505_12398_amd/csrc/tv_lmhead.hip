// LM head with fused row statistics for gfx950: logits = hidden * weight^T on
// bf16 MFMA, rounded to bf16, and in the same kernel the statistics of every
// row of the rounded logits that the verifier's tempered softmax needs (the
// row maximum and the sum of exp((z - max) / T)), so that no pass over the
// logits is needed to compute them (the distributions M_b and M_s of the
// problem statement, Alg. 3 REQUIRE, are softmax(logits / T) per row).
//
// Tiling. A workgroup of 256 threads (4 wavefronts, 2 x 2) computes a 128 x 128
// tile of logits; each wavefront a 64 x 64 sub-tile as 2 x 2 blocks of
// v_mfma_f32_32x32x16_bf16 (fp32 accumulation). K advances 64 at a time: the
// next K-slice of both operand tiles is loaded from global memory into
// registers (16-byte loads, coalesced along K) while the current one is
// multiplied from LDS. Both operands are K-contiguous (hidden [M][K], weight
// [N][K]), so every MFMA operand fragment is one 16-byte LDS read; LDS rows
// are padded by 16 bytes against bank conflicts. Each XCD gets a contiguous
// run of tiles, ordered in bands of 8 row tiles column tile by column tile,
// so the 8 x 8 or so tiles it runs at once read each slice of the hidden
// states and of the weight once from HBM and share it through the XCD's L2.
//
// Epilogue. Each accumulator is rounded to bf16 (round to nearest even) and
// stored. Per row, the wavefront reduces its 64 columns (max, then the sum of
// 2^((z - max) k), k = log2(e)/T, in fp32) across the 32 lanes that hold the
// row; the two wavefronts sharing a row merge through LDS; the workgroup
// writes one (max, sum) partial per row and column tile. A second kernel
// merges a row's partials in fp64 (exact power-of-two rescaling of each
// partial to the row maximum).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tv.h"
#include "tv_launch.h"

namespace {

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kLds = kBK + 8;          // padded LDS row, bf16 elements (144 bytes)
constexpr int kThreads = 256;
constexpr int kGroupM = 8;            // row tiles per band of the tile order

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

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet)
__device__ __forceinline__ uint16_t to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// One K-slice of a 128-row operand tile: 1024 16-byte vectors, four per
// thread (vector v = thread + 256 q: row v / 8, 8 bf16 at column 8 (v % 8)).
// Rows or columns outside the matrix read as zeros.
struct Slice {
  uint4 v[4];
  __device__ __forceinline__ void load(const uint16_t* base, int rows, int row0, int K, int k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = threadIdx.x + kThreads * q;
      const int r = row0 + (idx >> 3);
      const int c = k0 + 8 * (idx & 7);
      if (r < rows && c < K) {
        v[q] = *reinterpret_cast<const uint4*>(base + static_cast<size_t>(r) * K + c);
      } else {
        v[q] = make_uint4(0, 0, 0, 0);
      }
    }
  }
  __device__ __forceinline__ void store(uint16_t* lds) const {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = threadIdx.x + kThreads * q;
      *reinterpret_cast<uint4*>(lds + (idx >> 3) * kLds + 8 * (idx & 7)) = v[q];
    }
  }
};

__device__ __forceinline__ bf16x8 frag(const uint16_t* lds, int row, int k) {
  const uint4 u = *reinterpret_cast<const uint4*>(lds + row * kLds + k);
  return __builtin_bit_cast(bf16x8, u);
}

__global__ void __launch_bounds__(kThreads) lmhead_kernel(LmParams P) {
  __shared__ __attribute__((aligned(16))) uint16_t As[kBM * kLds];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[kBN * kLds];
  __shared__ float red_m[2][kBM];
  __shared__ float red_s[2][kBM];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  // Workgroups are dealt to the 8 XCDs in turn (workgroup i to XCD i % 8):
  // the remap gives each XCD a contiguous run of logical tiles (any grid
  // size), and the logical order walks bands of kGroupM row tiles column tile
  // by column tile, so the tiles an XCD runs at once form a block of about
  // kGroupM x kGroupM that shares each operand slice through its L2.
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

  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

  Slice sa, sb;
  sa.load(P.x, P.M, m0, P.K, 0);
  sb.load(P.w, P.N, n0, P.K, 0);
  const int lr = lane & 31, lh = lane >> 5;
  for (int k0 = 0; k0 < P.K; k0 += kBK) {
    __syncthreads();                 // the previous slice has been consumed
    sa.store(As);
    sb.store(Bs);
    __syncthreads();
    if (k0 + kBK < P.K) {            // next slice in flight during the products
      sa.load(P.x, P.M, m0, P.K, k0 + kBK);
      sb.load(P.w, P.N, n0, P.K, k0 + kBK);
    }
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 16) {
      bf16x8 fa[2], fb[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) fa[a] = frag(As, wm * 64 + a * 32 + lr, kk + 8 * lh);
#pragma unroll
      for (int b = 0; b < 2; ++b) fb[b] = frag(Bs, wn * 64 + b * 32 + lr, kk + 8 * lh);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[b], acc[a][b], 0, 0, 0);
    }
  }

  // Epilogue: accumulator r of block (a, b) holds row
  // m0 + 64 wm + 32 a + 8 (r / 4) + 4 lh + r % 4 and column n0 + 64 wn + 32 b + lr.
  const float k = P.k32;
  float zb[2][2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int col = n0 + wn * 64 + b * 32 + lr;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        const uint16_t h = to_bf16(acc[a][b][r]);
        if (row < P.M && col < P.N) P.logits[static_cast<size_t>(row) * P.N + col] = h;
        zb[a][b][r] = col < P.N ? bf16_to_f32(h) : -INFINITY;
      }
    }
  // row maxima over the wavefront's 64 columns: the two column blocks, then
  // the 32 lanes of this half of the wavefront
  float mx[2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float v = fmaxf(zb[a][0][r], zb[a][1][r]);
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
      mx[a][r] = v;
    }
  // sums of 2^((z - max) k) in the frame of the wavefront's row maximum (a
  // row whose maximum is -inf, every column masked or -inf, sums 0; NaN or
  // +inf propagate)
  float sm[2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float m = mx[a][r];
      const float c = (m > -INFINITY) ? -m * k : 0.0f;
      float v = 0.0f;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const float z = zb[a][b][r];
        v += (z > -INFINITY) ? __builtin_amdgcn_exp2f(fmaf(z, k, c)) : (z != z ? z : 0.0f);
      }
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) v += __shfl_xor(v, off, 64);
      sm[a][r] = v;
    }
  // the two wavefronts of a row band (wn = 0, 1) merge through LDS
  if (lr == 0) {
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wm * 64 + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        red_m[wn][rl] = mx[a][r];
        red_s[wn][rl] = sm[a][r];
      }
  }
  __syncthreads();
  if (tid < kBM) {
    const int row = m0 + tid;
    if (row < P.M) {
      const float ma = red_m[0][tid], mb = red_m[1][tid];
      const float sa_ = red_s[0][tid], sb_ = red_s[1][tid];
      const float m = fmaxf(ma, mb);
      float s;
      if (!(m > -INFINITY)) {
        s = sa_ + sb_;                                   // 0, or NaN
      } else {
        // frames -max * k as the terms used them (fp32 products)
        const float cm = -m * k;
        s = (ma > -INFINITY ? sa_ * __builtin_amdgcn_exp2f(cm - (-ma * k)) : sa_) +
            (mb > -INFINITY ? sb_ * __builtin_amdgcn_exp2f(cm - (-mb * k)) : sb_);
      }
      P.part_max[static_cast<size_t>(row) * P.tiles_n + tn] = m;
      P.part_sum[static_cast<size_t>(row) * P.tiles_n + tn] = s;
    }
  }
}

// Merges the column-tile partials of one row per wavefront (fp64 sum, each
// partial rescaled to the row maximum by an exact power of two).
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
  // row's frame -m * k by the exact power of two between the two frames
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
