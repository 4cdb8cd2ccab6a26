// MI355X (gfx950) kernels and C ABI of one Allegro layer around the tensor
// product.  What is computed is stated in include/allegro_layer.h.
//
// The dense contractions run on the fp32 matrix cores with
// v_mfma_f32_16x16x4_f32: for one instruction lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16], and accumulator register r of lane l holds
// D[4 (l / 16) + r][l % 16].  Over the steps of a sum, lane group l / 16
// either interleaves with the others (k = 4 s + l / 16) or owns a contiguous
// quarter of k, whichever keeps that kernel's LDS reads free of bank
// conflicts; A and B always use the same order, so every product pairs the
// same k.
//
//   row_gemm_kernel     C[E][N] = X[E][K] B[K][N], X = [x1 | x2] staged in LDS,
//                       with a fused prologue (SiLU) and epilogue (add,
//                       SiLU-gradient scale, column split): w = h A,
//                       a = [h, s] B1, h' = h + SiLU(a) B2 and their VJPs
//   reduce_gemm_kernel  G[M][N] = sum_e P[e][M] Q[e][N] (dA, dB1, dB2):
//                       persistent workgroups with register accumulators,
//                       one partial per workgroup, then colsum_kernel
//   mix_kernel          per-irrep channel mixing V' = Mix_c T_c (forward) or
//                       dT = Mix_c^T dV' (backward); each wave keeps its 16
//                       output channels' rows of every Mix_c in registers
//   mix_wgrad_kernel    dMix_c = sum over edges and components of dV'_c T_c^T
//   colsum_kernel       fixed-order sum of the workgroups' partials
//
// Edge-major [E][U][d1] tiles are staged through LDS in a per-irrep column
// layout: column (e, m) of irrep c holds the U channels of component
// off(c) + m of edge e, columns padded so that the 64 lanes of an MFMA
// operand read hit distinct banks.  All reductions over edges have a fixed
// order and no atomics, so every output is bit-identical run to run.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>

#include "allegro_layer.h"
#include "device_common.hpp"
#include "plan.hpp"

namespace {

using namespace allegro_dev;
using allegro_internal::fail;

constexpr int kWave = 64;
constexpr int kThreads = 256;  // four waves per workgroup
constexpr int kU = 64;         // channels supported by the layer

__device__ __forceinline__ f32x4 mfma_16x16x4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// SiLU(a) = a / (1 + exp(-a)) and its derivative sigma(a) (1 + a (1 - sigma(a))).
__device__ __forceinline__ float silu(float a) { return a / (1.0f + expf(-a)); }
__device__ __forceinline__ float silu_grad(float a) {
  const float sg = 1.0f / (1.0f + expf(-a));
  return sg * (1.0f + a * (1.0f - sg));
}

// The x irreps of a plan: for l = 0..lmax, (l, natural parity) then, with
// full parity, (l, the other parity); sizes 2l + 1, concatenated.
template <int LMAX, bool FULL>
struct XIrreps {
  static constexpr int NX = FULL ? 2 * (LMAX + 1) : LMAX + 1;
  static constexpr int D1 = FULL ? 2 * (LMAX + 1) * (LMAX + 1) : (LMAX + 1) * (LMAX + 1);
  static constexpr int dim(int c) { return 2 * (FULL ? c / 2 : c) + 1; }
  static constexpr int off(int c) { return c == 0 ? 0 : off(c - 1) + dim(c - 1); }
};

// ------------------------------------------------------------- row GEMM
enum { kProNone = 0, kProSilu = 1 };
enum { kEpiStore = 0, kEpiAdd = 1, kEpiSiluGrad = 2, kEpiSplitAdd = 3 };

struct RowGemmArgs {
  int64_t E;
  const float *x1, *x2;  // X = [x1 | x2], [E][K1] and [E][K2]
  const float *b;        // B[k][n] = b[k * b_rs + n * b_cs]
  int b_rs, b_cs;
  const float *d;        // addend (kEpiAdd, kEpiSplitAdd) or pre-activation (kEpiSiluGrad)
  float *c, *c2;         // output; kEpiSplitAdd: columns < N1 to c, the rest to c2
};

constexpr int kRowTile = 64;  // rows per workgroup tile

// Stages rows r0 .. r0 + 63 of x [E][KX] into columns col0 .. col0 + KX - 1 of
// the LDS tile (row stride XS), zero past the last row, with an optional
// elementwise prologue.  All of a thread's loads are issued before any of its
// LDS writes, so their latencies overlap.
template <int KX, int PRO>
__device__ __forceinline__ void stage_rows(const float *__restrict__ x, int64_t r0, int rows, float *xs, int XS,
                                           int col0, int tid) {
  constexpr int F4 = kRowTile * KX / 4, PER = (F4 + kThreads - 1) / kThreads;
  float4 v[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int f = tid + kThreads * i, r = f / (KX / 4), k = 4 * (f % (KX / 4));
    v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (f < F4 && r < rows) v[i] = *reinterpret_cast<const float4 *>(x + (r0 + r) * KX + k);
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int f = tid + kThreads * i, r = f / (KX / 4), k = 4 * (f % (KX / 4));
    if (f >= F4) continue;
    float4 u = v[i];
    if constexpr (PRO == kProSilu) {
      u.x = silu(u.x); u.y = silu(u.y); u.z = silu(u.z); u.w = silu(u.w);
    }
    *reinterpret_cast<float4 *>(xs + r * XS + col0 + k) = u;
  }
}

// stage_rows in two halves, so that a tile's loads can be in flight while the
// previous tile is multiplied: the loads into registers, then the LDS writes.
template <int KX>
struct RowRegs {
  static constexpr int F4 = kRowTile * KX / 4, PER = (F4 + kThreads - 1) / kThreads;
  float4 v[PER];
  __device__ __forceinline__ void load(const float *__restrict__ x, int64_t r0, int rows, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = tid + kThreads * i, r = f / (KX / 4), k = 4 * (f % (KX / 4));
      v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (f < F4 && r < rows) v[i] = *reinterpret_cast<const float4 *>(x + (r0 + r) * KX + k);
    }
  }
  template <int PRO>
  __device__ __forceinline__ void put(float *xs, int XS, int col0, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = tid + kThreads * i, r = f / (KX / 4), k = 4 * (f % (KX / 4));
      if (f >= F4) continue;
      float4 u = v[i];
      if constexpr (PRO == kProSilu) {
        u.x = silu(u.x); u.y = silu(u.y); u.z = silu(u.z); u.w = silu(u.w);
      }
      *reinterpret_cast<float4 *>(xs + r * XS + col0 + k) = u;
    }
  }
};

// C[E][N] = X[E][K] B[K][N] over 64-row tiles.  Wave w owns the column tiles
// w + 4 j of every row tile and keeps their B operands in registers for the
// whole launch; A operands come from the LDS tile.  The products of the tile
// go back through LDS (over the X tile), so that the epilogue reads its addend
// and writes its output as whole rows, 16 bytes per lane and consecutive
// lanes along a row: written straight from the accumulators, each store
// instruction would cover 64-byte pieces of four rows.
template <int K1, int K2, int N, int N1, int PRO, int EPI>
__global__ __launch_bounds__(kThreads) void row_gemm_kernel(RowGemmArgs g) {
  constexpr int K = K1 + K2, XS = K + 4;  // row stride: the 16 rows of an A read hit distinct banks
  constexpr int OS = N + 4;               // row stride of the product tile
  constexpr int NJ = N / 64;              // column tiles per wave
  constexpr int LDSF = kRowTile * (XS > OS ? XS : OS);
  constexpr int OF4 = kRowTile * N / 4, OPER = OF4 / kThreads;  // product float4 per thread
  static_assert(K1 % 16 == 0 && K2 % 16 == 0 && N % 64 == 0 && N1 % 16 == 0 && OF4 % kThreads == 0, "tile shape");
  __shared__ float4 xs4[LDSF / 4];
  float *xs = reinterpret_cast<float *>(xs4);
  const int tid = threadIdx.x, wave = tid / kWave, l = tid % kWave;
  // step s pairs k = 4 s + l / 16 in both operands
  float bf[NJ][K / 4];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int s = 0; s < K / 4; ++s)
      bf[j][s] = g.b[(4 * s + l / 16) * g.b_rs + (16 * (wave + 4 * j) + l % 16) * g.b_cs];
  const int64_t n_tiles = (g.E + kRowTile - 1) / kRowTile;
  // the next tile's rows are loaded while this tile is multiplied
  RowRegs<K1> x1r;
  RowRegs<(K2 > 0 ? K2 : 4)> x2r;
  auto load = [&](int64_t t) {
    const int64_t r0 = t * kRowTile;
    const int rows = int(g.E - r0 < kRowTile ? g.E - r0 : kRowTile);
    x1r.load(g.x1, r0, rows, tid);
    if constexpr (K2 > 0) x2r.load(g.x2, r0, rows, tid);
  };
  if (int64_t(blockIdx.x) < n_tiles) load(blockIdx.x);
  for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
    const int64_t r0 = t * kRowTile;
    const int rows = int(g.E - r0 < kRowTile ? g.E - r0 : kRowTile);
    x1r.template put<PRO>(xs, XS, 0, tid);
    if constexpr (K2 > 0) x2r.template put<kProNone>(xs, XS, K1, tid);
    lds_sync<4>();
    if (t + gridDim.x < n_tiles) load(t + gridDim.x);
    f32x4 acc[kRowTile / 16][NJ];
#pragma unroll
    for (int rt = 0; rt < kRowTile / 16; ++rt) {
      // with XS = 4 (mod 64) the 64 lanes of an A read hit distinct banks
      const float *xa = xs + (16 * rt + l % 16) * XS + l / 16;
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[rt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < K / 4; ++s) {
        const float a = xa[4 * s];
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[rt][j] = mfma_16x16x4(a, bf[j][s], acc[rt][j]);
      }
    }
    lds_sync<4>();  // every wave has read the X tile: its LDS takes the products
#pragma unroll
    for (int rt = 0; rt < kRowTile / 16; ++rt)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          xs[(16 * rt + 4 * (l / 16) + r) * OS + 16 * (wave + 4 * j) + l % 16] = acc[rt][j][r];
    lds_sync<4>();
    // epilogue by whole rows: float4 f = tid + 256 i is row f / (N / 4), columns 4 (f % (N / 4)) ..
    float4 dv[OPER];
    if constexpr (EPI != kEpiStore) {
#pragma unroll
      for (int i = 0; i < OPER; ++i) {
        const int f = tid + kThreads * i, row = f / (N / 4), col = 4 * (f % (N / 4));
        dv[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row < rows && (EPI != kEpiSplitAdd || col < N1)) {
          const int64_t e = r0 + row;
          dv[i] = *reinterpret_cast<const float4 *>(g.d + e * (EPI == kEpiSplitAdd ? N1 : N) + col);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < OPER; ++i) {
      const int f = tid + kThreads * i, row = f / (N / 4), col = 4 * (f % (N / 4));
      if (row >= rows) continue;
      const int64_t e = r0 + row;
      float4 v = *reinterpret_cast<const float4 *>(xs + row * OS + col);
      if constexpr (EPI == kEpiAdd) {
        v.x += dv[i].x; v.y += dv[i].y; v.z += dv[i].z; v.w += dv[i].w;
      } else if constexpr (EPI == kEpiSiluGrad) {
        v.x *= silu_grad(dv[i].x); v.y *= silu_grad(dv[i].y); v.z *= silu_grad(dv[i].z); v.w *= silu_grad(dv[i].w);
      }
      if constexpr (EPI == kEpiSplitAdd) {
        if (col < N1) {
          v.x += dv[i].x; v.y += dv[i].y; v.z += dv[i].z; v.w += dv[i].w;
          *reinterpret_cast<float4 *>(g.c + e * N1 + col) = v;
        } else {
          *reinterpret_cast<float4 *>(g.c2 + e * (N - N1) + (col - N1)) = v;
        }
      } else {
        *reinterpret_cast<float4 *>(g.c + e * N + col) = v;
      }
    }
    lds_sync<4>();  // the products are read: the next X tile may land
  }
}

// ---------------------------------------------------------- reduce GEMM
constexpr int kRedTile = 64;  // edges per step

template <int M1, int M2, int N, int PRO>
__global__ __launch_bounds__(kThreads) void reduce_gemm_kernel(int64_t E, const float *__restrict__ p1,
                                                               const float *__restrict__ p2,
                                                               const float *__restrict__ q,
                                                               float *__restrict__ part) {
  constexpr int M = M1 + M2, PS = M + 16, QS = N + 16;  // strides = 16 (mod 64): conflict-free operand reads
  constexpr int MT = M / 16, NJ = N / 64;  // wave w owns column tiles nt = w + 4 j (j < NJ) of every row tile
  static_assert(M1 % 16 == 0 && M2 % 16 == 0 && N % 64 == 0, "tile shape");
  __shared__ float4 ps4[kRedTile * PS / 4], qs4[kRedTile * QS / 4];
  float *ps = reinterpret_cast<float *>(ps4), *qs = reinterpret_cast<float *>(qs4);
  const int tid = threadIdx.x, wave = tid / kWave, l = tid % kWave;
  f32x4 acc[MT][NJ];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int64_t n_tiles = (E + kRedTile - 1) / kRedTile;
  static_assert(kRedTile == kRowTile, "tiles staged by RowRegs");
  // the next tile's loads are issued before this tile's products, into the
  // registers this tile's rows have just left
  RowRegs<M1> r1;
  RowRegs<(M2 > 0 ? M2 : 4)> r2;
  RowRegs<N> rq;
  auto load = [&](int64_t t) {
    const int64_t r0 = t * kRedTile;
    const int rows = int(E - r0 < kRedTile ? E - r0 : kRedTile);
    r1.load(p1, r0, rows, tid);
    if constexpr (M2 > 0) r2.load(p2, r0, rows, tid);
    rq.load(q, r0, rows, tid);
  };
  if (int64_t(blockIdx.x) < n_tiles) load(blockIdx.x);
  for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
    r1.template put<PRO>(ps, PS, 0, tid);
    if constexpr (M2 > 0) r2.template put<kProNone>(ps, PS, M1, tid);
    rq.template put<kProNone>(qs, QS, 0, tid);
    lds_sync<4>();
    if (t + gridDim.x < n_tiles) load(t + gridDim.x);
    // the sum runs over the tile's edges: step s pairs edge 4 s + l / 16
    const float *pa = ps + (l / 16) * PS + l % 16;
    const float *qb = qs + (l / 16) * QS + 16 * wave + l % 16;
#pragma unroll 2
    for (int s = 0; s < kRedTile / 4; ++s) {
      float a[MT], b[NJ];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) a[mt] = pa[4 * s * PS + 16 * mt];
#pragma unroll
      for (int j = 0; j < NJ; ++j) b[j] = qb[4 * s * QS + 64 * j];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[mt][j] = mfma_16x16x4(a[mt], b[j], acc[mt][j]);
    }
    lds_sync<4>();
  }
  float *out = part + int64_t(blockIdx.x) * M * N;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        out[(16 * mt + 4 * (l / 16) + r) * N + 16 * (wave + 4 * j) + l % 16] = acc[mt][j][r];
}

// out[c] = sum over r of part[r][c], in a fixed order: a block owns 16
// columns; thread (g, c) sums rows g, g + 16, g + 32, ... with four
// accumulators, then the 16 row groups are added in order.
constexpr int kColsumCols = 16, kColsumGroups = 16;

__global__ __launch_bounds__(256) void colsum_kernel(int R, int C, const float *__restrict__ part,
                                                     float *__restrict__ out) {
  __shared__ float sums[kColsumGroups][kColsumCols];
  const int cl = int(threadIdx.x) % kColsumCols, g = int(threadIdx.x) / kColsumCols;
  const int c = int(blockIdx.x) * kColsumCols + cl;
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  if (c < C) {
    int r = g;
    constexpr int S = kColsumGroups;
    for (; r + 3 * S < R; r += 4 * S) {
      a0 += part[int64_t(r) * C + c];
      a1 += part[int64_t(r + S) * C + c];
      a2 += part[int64_t(r + 2 * S) * C + c];
      a3 += part[int64_t(r + 3 * S) * C + c];
    }
    for (; r < R; r += S) a0 += part[int64_t(r) * C + c];
  }
  sums[g][cl] = (a0 + a1) + (a2 + a3);
  __syncthreads();
  if (g == 0 && c < C) {
    float a = sums[0][cl];
    for (int k = 1; k < kColsumGroups; ++k) a += sums[k][cl];
    out[c] = a;
  }
}

// ------------------------------------------------------------ mixing
// LDS column index of component k of edge e in a tile of ne_tile edges.
template <class X>
__device__ __forceinline__ void component_column(int k, int ne_tile, int &col0, int &dim) {
  int c = 0;
#pragma unroll
  for (int i = 1; i < X::NX; ++i) c = k >= X::off(i) ? i : c;
  int o = 0, d = 1;
#pragma unroll
  for (int i = 0; i < X::NX; ++i)
    if (i == c) { o = X::off(i); d = X::dim(i); }
  col0 = ne_tile * o + (k - o);
  dim = d;
}

constexpr int kMixEdges = 8;       // edges per tile
// Column stride (floats): a multiple of 4, so a lane reads its 16 B operands
// of a step block as four 16-byte LDS loads, and 68 = 4 (mod 64), so the 16
// columns of a tile start in distinct bank quads.
constexpr int kMixCS = kU + 4;
constexpr int kMixThreads = 512;   // four compute waves, then four memory waves

// Per-irrep channel mixing, software-pipelined over two LDS tile buffers.
// Waves 0-3 (compute) hold rows 16w .. 16w+15 of every Mix_c (Mix_c^T for the
// backward) in registers and run the matrix-core products on one buffer,
// while waves 4-7 (memory) store the previous tile's results from the other
// buffer and refill it with the next tile.  Per tile the two roles meet at
// two workgroup barriers: after the first the compute waves write their
// results into their buffer in place, after the second the buffers swap.
// Both roles run the same tile sequence, so their barrier counts match.
template <class X>
struct MixTile {
  static constexpr int U = kU, D1 = X::D1, NX = X::NX, NE = kMixEdges, CS = kMixCS;
  static constexpr int COLS = NE * D1;
  static constexpr int BUF = (COLS + 16) * CS;  // +16 columns: the last irrep's padded column tile
  static constexpr int F4 = NE * U * D1 / 4;    // float4 per full tile
  static constexpr int PER = (F4 + 255) / 256;  // float4 per memory thread
  static constexpr int ncols(int c) { return NE * X::dim(c); }
  static constexpr int nct(int c) { return (ncols(c) + 15) / 16; }
  static constexpr int ct_off(int c) { return c == 0 ? 0 : ct_off(c - 1) + nct(c - 1); }
  static constexpr int NCT = ct_off(NX);
  static_assert((U * D1) % 4 == 0, "edge rows must be whole float4");
  static_assert(CS % 4 == 0, "operand blocks are read as 16-byte LDS loads");
};

template <class X, bool BWD>
__device__ __forceinline__ void mix_compute_role(int64_t E, int64_t n_tiles, const float *__restrict__ mix,
                                                 const float *__restrict__ ds, float *__restrict__ s_out,
                                                 float *lds) {
  using M = MixTile<X>;
  constexpr int U = M::U, CS = M::CS, NE = M::NE;
  const int tid = threadIdx.x, w = tid / kWave, l = tid % kWave;
  // A operands: row 16 w + l % 16 of Mix_c (or of Mix_c^T), columns 16 (l / 16) + s
  float A[M::NX][16];
  static_for<0, M::NX>([&](auto ic) {
    constexpr int c = decltype(ic)::value;
#pragma unroll
    for (int s = 0; s < 16; ++s)
      A[c][s] = BWD ? mix[(c * U + 16 * (l / 16) + s) * U + 16 * w + l % 16]
                    : mix[(c * U + 16 * w + l % 16) * U + 16 * (l / 16) + s];
  });
  lds_sync<8>();  // the first tile is in buffer 0
  int p = 0;
  for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x, ++p) {
    float *b = lds + (p & 1) * M::BUF;
    const int64_t e0 = t * NE;
    const int ne = int(E - e0 < NE ? E - e0 : NE);
    // backward: the lane's ds terms for the 0e columns (column q = edge q), loaded
    // now so that their latency hides under the products
    float dsv[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (BWD) {
      if (l % 16 < ne) {
#pragma unroll
        for (int r = 0; r < 4; ++r) dsv[r] = ds[(e0 + l % 16) * U + 16 * w + 4 * (l / 16) + r];
      }
    }
    f32x4 acc[M::NCT];
    static_for<0, M::NX>([&](auto ic) {
      constexpr int c = decltype(ic)::value, base = NE * X::off(c);
#pragma unroll
      for (int ct = 0; ct < M::nct(c); ++ct) {
        // the lane's 16 operands (channels 16 (l / 16) .. + 15 of column 16 ct + l % 16) are contiguous
        const float4 *bp = reinterpret_cast<const float4 *>(b + (base + 16 * ct + l % 16) * CS + 16 * (l / 16));
        float bv[16];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float4 x = bp[j];
          bv[4 * j] = x.x; bv[4 * j + 1] = x.y; bv[4 * j + 2] = x.z; bv[4 * j + 3] = x.w;
        }
        f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 16; ++s) a = mfma_16x16x4(A[c][s], bv[s], a);
        acc[M::ct_off(c) + ct] = a;
      }
    });
    if constexpr (!BWD) {
      // s[e][u] = T[e][u][0]: irrep 0 (0e) has one component, so its column is e
      for (int i = tid; i < ne * U; i += 256) s_out[(e0 + i / U) * U + i % U] = b[(i / U) * CS + i % U];
    }
    lds_sync<8>();  // B1: every compute wave has read the tile
    static_for<0, M::NX>([&](auto ic) {
      constexpr int c = decltype(ic)::value, base = NE * X::off(c), nq = M::ncols(c);
#pragma unroll
      for (int ct = 0; ct < M::nct(c); ++ct) {
        const int q = 16 * ct + l % 16;
        if (q >= nq) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int uo = 16 * w + 4 * (l / 16) + r;
          float val = acc[M::ct_off(c) + ct][r];
          if constexpr (BWD && c == 0) val += dsv[r];  // zero for columns past the tile's edges
          b[(base + q) * CS + uo] = val;
        }
      }
    });
    lds_sync<8>();  // B2: results are in the buffer
  }
}

template <class X>
__device__ __forceinline__ void mix_memory_role(int64_t E, int64_t n_tiles, const float *__restrict__ src,
                                                float *__restrict__ dst, float *lds) {
  using M = MixTile<X>;
  constexpr int U = M::U, D1 = M::D1, NE = M::NE, PER = M::PER, F4 = M::F4;
  const int mt = int(threadIdx.x) - 256;
  // The thread's float4 of a tile: fi(i) = f0 + 16 i.  Each group of 16 lanes
  // covers 256 contiguous bytes per access (coalesced), and a thread's float4
  // lie 256 B apart, within the reach of one base address and immediate
  // offsets (4 KB apart, as with fi(i) = mt + 256 i, measured 4% slower).
  const int f0 = (mt / 16) * (16 * PER) + mt % 16;
  auto fi = [&](int i) { return f0 + 16 * i; };
  // LDS offset (within a buffer) of each of the thread's elements: component k
  // of channel u of edge e sits in column NE off(c) + e dim(c) + m, row u
  int addr[PER][4];
#pragma unroll
  for (int i = 0; i < PER; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = 4 * fi(i) + q;
      int a = 0;
      if (idx < 4 * F4) {
        const int e = idx / (U * D1), rem = idx % (U * D1), u = rem / D1, k = rem % D1;
        int col0, dim;
        component_column<X>(k, NE, col0, dim);
        a = (col0 + e * dim) * M::CS + u;
      }
      addr[i][q] = a;
    }
  auto count = [&](int64_t t) { return int(E - t * NE < NE ? E - t * NE : NE) * (U * D1 / 4); };
  auto load = [&](int64_t t, float4 (&v)[PER]) {
    const int nf4 = count(t);
    const float4 *s4 = reinterpret_cast<const float4 *>(src + t * NE * U * D1);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = fi(i);
      v[i] = f < nf4 ? load_stream(s4 + f) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto put = [&](float *b, const float4 (&v)[PER]) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (fi(i) >= F4) continue;
      b[addr[i][0]] = v[i].x;
      b[addr[i][1]] = v[i].y;
      b[addr[i][2]] = v[i].z;
      b[addr[i][3]] = v[i].w;
    }
  };
  auto store = [&](int64_t t, const float *b) {
    const int nf4 = count(t);
    float4 *d4 = reinterpret_cast<float4 *>(dst + t * NE * U * D1);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = fi(i);
      if (f < nf4) store_stream(make_float4(b[addr[i][0]], b[addr[i][1]], b[addr[i][2]], b[addr[i][3]]), d4 + f);
    }
  };
  // The tile after the next one is loaded into registers one period ahead,
  // so its loads stay in flight across the barriers and the compute waves'
  // write-back.
  const int64_t G = gridDim.x;
  int64_t t = blockIdx.x;
  float4 v[PER];
  if (t < n_tiles) {
    load(t, v);
    put(lds, v);
  }
  if (t + G < n_tiles) load(t + G, v);
  lds_sync<8>();
  int p = 0;
  for (; t < n_tiles; t += G, ++p) {
    // each LDS element is read (store of tile t - G) and then overwritten (tile
    // t + G) by the same thread, so program order alone orders the two
    float *b = lds + ((p + 1) & 1) * M::BUF;
    if (p > 0) store(t - G, b);
    if (t + G < n_tiles) put(b, v);
    if (t + 2 * G < n_tiles) load(t + 2 * G, v);
    lds_sync<8>();  // B1
    lds_sync<8>();  // B2: the compute waves have written tile t's results
  }
  if (p > 0) store(t - G, lds + ((p + 1) & 1) * M::BUF);
}

template <int LMAX, bool FULL, bool BWD>
__global__ __launch_bounds__(kMixThreads) void mix_kernel(int64_t E, const float *__restrict__ src,
                                                          const float *__restrict__ mix,
                                                          const float *__restrict__ ds, float *__restrict__ dst,
                                                          float *__restrict__ s_out) {
  using X = XIrreps<LMAX, FULL>;
  __shared__ float lds[2 * MixTile<X>::BUF];
  const int64_t n_tiles = (E + kMixEdges - 1) / kMixEdges;
  if (threadIdx.x < 256) mix_compute_role<X, BWD>(E, n_tiles, mix, ds, s_out, lds);
  else mix_memory_role<X>(E, n_tiles, src, dst, lds);
}

constexpr int kWgEdges = 4;        // edges per tile: column counts NE * (2l + 1) are multiples of 4
// Channel u of the column of component k sits at u ^ wg_swizzle(k) (bits 1-3,
// within its 16-channel block).  A memory wave's 4-byte writes of one
// instruction cover 8 components k = 4 b + q (b = 0..7) of up to 8 channels;
// the swizzle spreads them over 64 distinct banks (without it 8 lanes shared
// a bank), and the compute waves' reads of 16 consecutive channels of one
// column stay a permutation of one 16-bank block.
__host__ __device__ constexpr int wg_swizzle(int k) { return 2 * (k >> 2); }
constexpr int kWgCS = kU + 16;     // = 16 (mod 64): the four lane groups of an operand read hit distinct banks
constexpr int kWgThreads = 512;    // four compute waves, then four memory waves

// dMix_c = sum over edges and components of dV'_c T_c^T, software-pipelined
// over two LDS buffers that each hold a tile of dV' and of T in the column
// layout of the mixing kernel.  Waves 0-3 (compute) own rows 16w .. 16w+15 of
// every dMix_c as register accumulators; waves 4-7 (memory) keep the next tile
// in registers and move it into the free buffer while the compute waves work
// on the other.  One barrier per tile; both roles run the same tile sequence.
// Each workgroup writes one partial of every dMix_c.
template <class X>
struct WgTile {
  static constexpr int U = kU, D1 = X::D1, NE = kWgEdges, CS = kWgCS;
  static constexpr int COLS = NE * D1;
  static constexpr int BUF = 2 * COLS * CS;     // dV' then T
  static constexpr int F4 = NE * U * D1 / 4;    // float4 per tensor and tile
  static constexpr int PER = (F4 + 255) / 256;  // float4 per memory thread and tensor
  static_assert((U * D1) % 4 == 0, "edge rows must be whole float4");
};

template <class X>
__device__ __forceinline__ void wgrad_compute_role(int64_t n_tiles, float *lds, float *__restrict__ part) {
  using M = WgTile<X>;
  constexpr int U = M::U, CS = M::CS, NE = M::NE, NX = X::NX;
  const int tid = threadIdx.x, w = tid / kWave, l = tid % kWave;
  f32x4 acc[NX][4];
#pragma unroll
  for (int c = 0; c < NX; ++c)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[c][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  lds_sync<8>();  // the first tile is in buffer 0
  int p = 0;
  for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x, ++p) {
    const float *la = lds + (p & 1) * M::BUF, *lb = la + M::COLS * CS;
    // dMix_c[v][u] += sum_q dV'_c[q][v] T_c[q][u]; lane group l / 16 owns
    // the quarter of the irrep's columns q = (l / 16) * nq / 4 + s
    static_for<0, NX>([&](auto ic) {
      constexpr int c = decltype(ic)::value, nq = NE * X::dim(c), base = NE * X::off(c);
      const int q0 = base + (l / 16) * (nq / 4);
#pragma unroll
      for (int s = 0; s < nq / 4; ++s) {
        // column q0 + s holds component off(c) + s (of edge l / 16): its
        // channels sit XOR-swizzled by wg_swizzle of that component
        const int ul = (l % 16) ^ wg_swizzle(X::off(c) + s);
        const float a = la[(q0 + s) * CS + 16 * w + ul];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) acc[c][nt] = mfma_16x16x4(a, lb[(q0 + s) * CS + 16 * nt + ul], acc[c][nt]);
      }
    });
    lds_sync<8>();  // this buffer is free again; the other holds the next tile
  }
  float *out = part + int64_t(blockIdx.x) * NX * U * U;
#pragma unroll
  for (int c = 0; c < NX; ++c)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        out[(c * U + 16 * w + 4 * (l / 16) + r) * U + 16 * nt + l % 16] = acc[c][nt][r];
}

template <class X>
__device__ __forceinline__ void wgrad_memory_role(int64_t E, int64_t n_tiles, const float *__restrict__ dv,
                                                  const float *__restrict__ tt, float *lds) {
  using M = WgTile<X>;
  constexpr int U = M::U, D1 = M::D1, NE = M::NE, PER = M::PER, F4 = M::F4;
  const int mt = int(threadIdx.x) - 256;
  // the thread's float4 of a tile, 256 B apart (as in mix_memory_role)
  const int f0 = (mt / 16) * (16 * PER) + mt % 16;
  auto fi = [&](int i) { return f0 + 16 * i; };
  // LDS offset (within a tensor's tile) of each of the thread's elements
  int addr[PER][4];
#pragma unroll
  for (int i = 0; i < PER; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = 4 * fi(i) + q;
      int a = 0;
      if (idx < 4 * F4) {
        const int e = idx / (U * D1), rem = idx % (U * D1), u = rem / D1, k = rem % D1;
        int col0, dim;
        component_column<X>(k, NE, col0, dim);
        a = (col0 + e * dim) * M::CS + (u ^ wg_swizzle(k));
      }
      addr[i][q] = a;
    }
  float4 va[PER], vb[PER];
  auto load = [&](int64_t t) {
    const int nf4 = int(E - t * NE < NE ? E - t * NE : NE) * (U * D1 / 4);
    const float4 *a4 = reinterpret_cast<const float4 *>(dv + t * NE * U * D1);
    const float4 *b4 = reinterpret_cast<const float4 *>(tt + t * NE * U * D1);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = fi(i);
      va[i] = f < nf4 ? load_stream(a4 + f) : make_float4(0.f, 0.f, 0.f, 0.f);
      vb[i] = f < nf4 ? load_stream(b4 + f) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto put = [&](float *b) {
    float *la = b, *lb = b + M::COLS * M::CS;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (fi(i) >= F4) continue;
      la[addr[i][0]] = va[i].x; la[addr[i][1]] = va[i].y; la[addr[i][2]] = va[i].z; la[addr[i][3]] = va[i].w;
      lb[addr[i][0]] = vb[i].x; lb[addr[i][1]] = vb[i].y; lb[addr[i][2]] = vb[i].z; lb[addr[i][3]] = vb[i].w;
    }
  };
  const int64_t G = gridDim.x;
  int64_t t = blockIdx.x;
  if (t < n_tiles) {
    load(t);
    put(lds);
  }
  if (t + G < n_tiles) load(t + G);
  lds_sync<8>();
  for (int p = 0; t < n_tiles; t += G, ++p) {
    // the compute waves read buffer p & 1; fill the other with tile t + G, then
    // start the loads of tile t + 2G
    if (t + G < n_tiles) put(lds + ((p + 1) & 1) * M::BUF);
    if (t + 2 * G < n_tiles) load(t + 2 * G);
    lds_sync<8>();
  }
}

template <int LMAX, bool FULL>
__global__ __launch_bounds__(kWgThreads) void mix_wgrad_kernel(int64_t E, const float *__restrict__ dv,
                                                               const float *__restrict__ tt,
                                                               float *__restrict__ part) {
  using X = XIrreps<LMAX, FULL>;
  __shared__ float lds[2 * WgTile<X>::BUF];
  const int64_t n_tiles = (E + kWgEdges - 1) / kWgEdges;
  if (threadIdx.x < 256) wgrad_compute_role<X>(n_tiles, lds, part);
  else wgrad_memory_role<X>(E, n_tiles, dv, tt, lds);
}

// ------------------------------------------------------------- host side
constexpr int64_t kMaxPersistent = 512;  // workgroups of the persistent kernels (2 per CU)

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align256(size_t b) { return (b + 255) & ~size_t(255); }
int64_t red_groups(int64_t E) { return std::min<int64_t>(cdiv(E, kRedTile), kMaxPersistent); }
int64_t wgrad_groups(int64_t E) { return std::min<int64_t>(cdiv(E, kWgEdges), kMaxPersistent); }

struct Shape {
  int L = 0, H = 0, U = 0, d1 = 0, d2 = 0, P = 0, NX = 0;
  int64_t N = 0, E = 0;
};

// Byte offsets of the regions of the saved and workspace buffers.
struct SavedLayout {
  size_t w, env, T, s, a, total;
};
struct WorkLayout {
  size_t dT, da, dhm, ds, dw, genv, tpws, red, mixp, total, tpws_bytes;
};

SavedLayout saved_layout(const Shape &z) {
  SavedLayout o{};
  size_t at = 0;
  auto take = [&](size_t floats) { const size_t off = at; at += align256(floats * sizeof(float)); return off; };
  o.w = take(size_t(z.E) * z.U);
  o.env = take(size_t(z.N) * z.U * z.d2);
  o.T = take(size_t(z.E) * z.U * z.d1);
  o.s = take(size_t(z.E) * z.U);
  o.a = take(size_t(z.E) * z.H);
  o.total = at;
  return o;
}

WorkLayout work_layout(const allegro_tp_plan *plan, const Shape &z) {
  WorkLayout o{};
  size_t at = 0;
  auto take = [&](size_t bytes) { const size_t off = at; at += align256(bytes); return off; };
  const size_t f = sizeof(float);
  o.dT = take(size_t(z.E) * z.U * z.d1 * f);
  o.da = take(size_t(z.E) * z.H * f);
  o.dhm = take(size_t(z.E) * z.L * f);
  o.ds = take(size_t(z.E) * z.U * f);
  o.dw = take(size_t(z.E) * z.U * f);
  o.genv = take(size_t(z.N) * z.U * z.d2 * f);
  size_t tpws = 0;
  (void)allegro_tp_backward_workspace(plan, z.N, &tpws);
  o.tpws_bytes = tpws;
  o.tpws = take(tpws);
  const size_t mn = std::max({size_t(z.L + z.U) * z.H, size_t(z.H) * z.L, size_t(z.L) * z.U});
  o.red = take(size_t(red_groups(z.E)) * mn * f);
  o.mixp = take(size_t(wgrad_groups(z.E)) * z.NX * z.U * z.U * f);
  o.total = at;
  return o;
}

int after(const char *what) {
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(ALLEGRO_E_HIP, "%s launch failed: %s", what, hipGetErrorString(err));
  return ALLEGRO_OK;
}

// Workgroups of `kernel` (static LDS only) that the device holds at once; at
// least one per compute unit.
int64_t resident_groups(const void *kernel, int threads) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess || per_cu <= 0)
    per_cu = 1;
  return int64_t(cus) * per_cu;
}

void colsum(hipStream_t s, int64_t R, int C, const float *part, float *out) {
  hipLaunchKernelGGL(colsum_kernel, dim3(unsigned(cdiv(C, kColsumCols))), dim3(256), 0, s, int(R), C, part, out);
}

// Launchers of the dense contractions of a layer with latent width L and hidden width H.
template <int L, int H>
struct DenseOps {
  static constexpr int U = kU;
  // one workgroup per slot the GPU holds at once: each loads its B operands once
  template <int K1, int K2, int N, int N1, int PRO, int EPI>
  static void row(hipStream_t s, const RowGemmArgs &g) {
    if (g.E == 0) return;
    static const int64_t slots =
        resident_groups(reinterpret_cast<const void *>(&row_gemm_kernel<K1, K2, N, N1, PRO, EPI>), kThreads);
    const unsigned G = unsigned(std::min<int64_t>(cdiv(g.E, kRowTile), slots));
    hipLaunchKernelGGL((row_gemm_kernel<K1, K2, N, N1, PRO, EPI>), dim3(G), dim3(kThreads), 0, s, g);
  }
  template <int M1, int M2, int N, int PRO>
  static void reduce(hipStream_t s, int64_t E, const float *p1, const float *p2, const float *q, float *part,
                     float *out) {
    const int64_t G = red_groups(E);
    if (G > 0)
      hipLaunchKernelGGL((reduce_gemm_kernel<M1, M2, N, PRO>), dim3(unsigned(G)), dim3(kThreads), 0, s, E, p1, p2, q,
                         part);
    colsum(s, G, (M1 + M2) * N, part, out);
  }

  // w = h A;  a = [h, s] B1 (after the mixing has written s);  h' = h + SiLU(a) B2
  static void embed_weights(hipStream_t s, int64_t E, const float *h, const float *A, float *w) {
    row<L, 0, U, 0, kProNone, kEpiStore>(s, {E, h, nullptr, A, U, 1, nullptr, w, nullptr});
  }
  static void latent(hipStream_t s, int64_t E, const float *h, const float *sv, const float *B1, const float *B2,
                     float *a, float *h_out) {
    row<L, U, H, 0, kProNone, kEpiStore>(s, {E, h, sv, B1, H, 1, nullptr, a, nullptr});
    row<H, 0, L, 0, kProSilu, kEpiAdd>(s, {E, a, nullptr, B2, L, 1, h, h_out, nullptr});
  }
  // da = (dh' B2^T) * SiLU'(a);  [dhm | ds] = [dh', 0] + da B1^T;  dB2, dB1
  static void latent_vjp(hipStream_t s, int64_t E, const float *h, const float *sv, const float *a,
                         const float *B1, const float *B2, const float *dh_out, float *da, float *dhm, float *ds,
                         float *part, float *dB1, float *dB2) {
    row<L, 0, H, 0, kProNone, kEpiSiluGrad>(s, {E, dh_out, nullptr, B2, 1, L, a, da, nullptr});
    row<H, 0, L + U, L, kProNone, kEpiSplitAdd>(s, {E, da, nullptr, B1, 1, H, dh_out, dhm, ds});
    reduce<H, 0, L, kProSilu>(s, E, a, nullptr, dh_out, part, dB2);
    reduce<L, U, H, kProNone>(s, E, h, sv, da, part, dB1);
  }
  // dA = h^T dw;  dh = dhm + dw A^T
  static void embed_vjp(hipStream_t s, int64_t E, const float *h, const float *A, const float *dw, const float *dhm,
                        float *part, float *dA, float *dh) {
    reduce<L, 0, U, kProNone>(s, E, h, nullptr, dw, part, dA);
    row<U, 0, L, 0, kProNone, kEpiAdd>(s, {E, dw, nullptr, A, 1, U, dhm, dh, nullptr});
  }
};

struct DenseTable {
  void (*embed_weights)(hipStream_t, int64_t, const float *, const float *, float *) = nullptr;
  void (*latent)(hipStream_t, int64_t, const float *, const float *, const float *, const float *, float *,
                 float *) = nullptr;
  void (*latent_vjp)(hipStream_t, int64_t, const float *, const float *, const float *, const float *,
                     const float *, const float *, float *, float *, float *, float *, float *, float *) = nullptr;
  void (*embed_vjp)(hipStream_t, int64_t, const float *, const float *, const float *, const float *, float *,
                    float *, float *) = nullptr;
};

template <int L, int H>
DenseTable dense_table() {
  using D = DenseOps<L, H>;
  return {&D::embed_weights, &D::latent, &D::latent_vjp, &D::embed_vjp};
}

DenseTable select_dense(int L, int H) {
  if (L == 64 && H == 64) return dense_table<64, 64>();
  if (L == 64 && H == 128) return dense_table<64, 128>();
  if (L == 128 && H == 64) return dense_table<128, 64>();
  if (L == 128 && H == 128) return dense_table<128, 128>();
  return {};
}

// Launchers of the mixing kernels of one (lmax, parity).
template <int LMAX, bool FULL>
struct MixOps {
  // one workgroup per tile slot the GPU holds at once: each streams a fixed tile sequence
  template <bool BWD>
  static unsigned grid(int64_t E) {
    static const int64_t slots = resident_groups(reinterpret_cast<const void *>(&mix_kernel<LMAX, FULL, BWD>),
                                                 kMixThreads);
    return unsigned(std::min<int64_t>(cdiv(E, kMixEdges), slots));
  }
  static void forward(hipStream_t s, int64_t E, const float *T, const float *mix, float *V_out, float *sv) {
    if (E == 0) return;
    hipLaunchKernelGGL((mix_kernel<LMAX, FULL, false>), dim3(grid<false>(E)), dim3(kMixThreads), 0, s, E, T, mix,
                       nullptr, V_out, sv);
  }
  static void backward(hipStream_t s, int64_t E, const float *dV_out, const float *T, const float *mix,
                       const float *ds, float *dT, float *part, float *dmix) {
    using X = XIrreps<LMAX, FULL>;
    // resident workgroups (one per compute unit), at most the partials the workspace holds
    static const int64_t slots = std::min<int64_t>(
        resident_groups(reinterpret_cast<const void *>(&mix_wgrad_kernel<LMAX, FULL>), kWgThreads), kMaxPersistent);
    const int64_t Gw = std::min<int64_t>(wgrad_groups(E), slots);
    if (E > 0) {
      hipLaunchKernelGGL((mix_kernel<LMAX, FULL, true>), dim3(grid<true>(E)), dim3(kMixThreads), 0, s, E, dV_out,
                         mix, ds, dT, nullptr);
      hipLaunchKernelGGL((mix_wgrad_kernel<LMAX, FULL>), dim3(unsigned(Gw)), dim3(kWgThreads), 0, s, E, dV_out, T,
                         part);
    }
    colsum(s, Gw, X::NX * kU * kU, part, dmix);
  }
};

struct MixTable {
  void (*forward)(hipStream_t, int64_t, const float *, const float *, float *, float *) = nullptr;
  void (*backward)(hipStream_t, int64_t, const float *, const float *, const float *, const float *, float *,
                   float *, float *) = nullptr;
};

template <int LMAX, bool FULL>
MixTable mix_table() {
  return {&MixOps<LMAX, FULL>::forward, &MixOps<LMAX, FULL>::backward};
}

MixTable select_mix(int lmax, bool full) {
  switch (lmax * 2 + (full ? 1 : 0)) {
    case 2: return mix_table<1, false>();
    case 3: return mix_table<1, true>();
    case 4: return mix_table<2, false>();
    case 5: return mix_table<2, true>();
    case 6: return mix_table<3, false>();
    case 7: return mix_table<3, true>();
    default: return {};
  }
}

int layer_shape(const allegro_tp_plan *plan, int L, int H, int64_t N, int64_t E, Shape &z) {
  if (!plan) return fail(ALLEGRO_E_INVALID, "plan is NULL");
  if (N < 0 || E < 0) return fail(ALLEGRO_E_INVALID, "negative size (N=%lld, E=%lld)", (long long)N, (long long)E);
  if (N == 0 && E > 0) return fail(ALLEGRO_E_INVALID, "E=%lld edges but N=0 centers", (long long)E);
  if (N >= (int64_t(1) << 31)) return fail(ALLEGRO_E_INVALID, "N=%lld exceeds 2^31-1", (long long)N);
  if (plan->U != kU) return fail(ALLEGRO_E_UNSUPPORTED, "the layer supports U=64 (plan has U=%d)", plan->U);
  if (!select_dense(L, H).latent)
    return fail(ALLEGRO_E_UNSUPPORTED, "the layer supports L, H in {64, 128} (got L=%d, H=%d)", L, H);
  const auto &t = plan->table;
  z.L = L;
  z.H = H;
  z.U = plan->U;
  z.d1 = t.d1;
  z.d2 = t.d2;
  z.P = int(t.paths.size());
  z.NX = int(t.x_irreps.size());
  z.N = N;
  z.E = E;
  return ALLEGRO_OK;
}

int check_ptr(const void *p, const char *name) {
  if (!p) return fail(ALLEGRO_E_INVALID, "%s is NULL", name);
  if (reinterpret_cast<uintptr_t>(p) & 15u) return fail(ALLEGRO_E_INVALID, "%s is not 16-byte aligned", name);
  return ALLEGRO_OK;
}

template <class T>
T *at(void *base, size_t off) {
  return reinterpret_cast<T *>(static_cast<char *>(base) + off);
}

}  // namespace

extern "C" {

int allegro_layer_buffers(const allegro_tp_plan *plan, int L, int H, int64_t N, int64_t E, size_t *saved_bytes,
                          size_t *workspace_bytes) {
  Shape z;
  int rc = layer_shape(plan, L, H, N, E, z);
  if (rc) return rc;
  if (saved_bytes) *saved_bytes = saved_layout(z).total;
  if (workspace_bytes) *workspace_bytes = work_layout(plan, z).total;
  return ALLEGRO_OK;
}

int allegro_layer_forward(const allegro_tp_plan *plan, int L, int H, int64_t N, int64_t E, const int64_t *row_ptr,
                          const float *h, const float *V, const float *Y, const float *A, const float *W,
                          const float *Mix, const float *B1, const float *B2, float *h_out, float *V_out,
                          void *saved, size_t saved_bytes, void *stream) {
  Shape z;
  int rc = layer_shape(plan, L, H, N, E, z);
  if (rc) return rc;
  if (N == 0) return ALLEGRO_OK;
  const SavedLayout sl = saved_layout(z);
  if ((rc = check_ptr(saved, "saved"))) return rc;
  if (saved_bytes < sl.total)
    return fail(ALLEGRO_E_INVALID, "saved buffer of %zu bytes is smaller than the %zu required", saved_bytes,
                sl.total);
  if ((rc = check_ptr(W, "W")) || (rc = check_ptr(A, "A")) || (rc = check_ptr(Mix, "Mix")) ||
      (rc = check_ptr(B1, "B1")) || (rc = check_ptr(B2, "B2")))
    return rc;
  if (E > 0 && ((rc = check_ptr(h, "h")) || (rc = check_ptr(V, "V")) || (rc = check_ptr(Y, "Y")) ||
                (rc = check_ptr(h_out, "h_out")) || (rc = check_ptr(V_out, "V_out"))))
    return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const DenseTable dn = select_dense(L, H);
  const MixTable mx = select_mix(plan->lmax, (plan->flags & ALLEGRO_FULL_PARITY) != 0);
  if (!mx.forward) return fail(ALLEGRO_E_UNSUPPORTED, "no mixing kernel for this plan");
  float *w = at<float>(saved, sl.w), *env = at<float>(saved, sl.env), *T = at<float>(saved, sl.T);
  float *sv = at<float>(saved, sl.s), *a = at<float>(saved, sl.a);
  dn.embed_weights(s, E, h, A, w);
  if ((rc = after("allegro_layer_forward"))) return rc;
  if ((rc = allegro_env_embed(plan, N, E, row_ptr, w, Y, env, stream))) return rc;
  if ((rc = allegro_tp_forward(plan, N, E, row_ptr, V, env, W, T, stream))) return rc;
  mx.forward(s, E, T, Mix, V_out, sv);
  dn.latent(s, E, h, sv, B1, B2, a, h_out);
  return after("allegro_layer_forward");
}

int allegro_layer_backward(const allegro_tp_plan *plan, int L, int H, int64_t N, int64_t E, const int64_t *row_ptr,
                           const float *h, const float *V, const float *Y, const float *A, const float *W,
                           const float *Mix, const float *B1, const float *B2, const void *saved, size_t saved_bytes,
                           const float *dh_out, const float *dV_out, float *dh, float *dV, float *dY, float *dA,
                           float *dW, float *dMix, float *dB1, float *dB2, void *workspace, size_t workspace_bytes,
                           void *stream) {
  Shape z;
  int rc = layer_shape(plan, L, H, N, E, z);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((rc = check_ptr(dA, "dA")) || (rc = check_ptr(dW, "dW")) || (rc = check_ptr(dMix, "dMix")) ||
      (rc = check_ptr(dB1, "dB1")) || (rc = check_ptr(dB2, "dB2")) || (rc = check_ptr(W, "W")) ||
      (rc = check_ptr(A, "A")) || (rc = check_ptr(Mix, "Mix")) || (rc = check_ptr(B1, "B1")) ||
      (rc = check_ptr(B2, "B2")))
    return rc;
  if (N == 0) {  // no centers, no edges: every weight gradient is zero
    colsum(s, 0, z.L * z.U, nullptr, dA);
    colsum(s, 0, z.P * z.U, nullptr, dW);
    colsum(s, 0, z.NX * z.U * z.U, nullptr, dMix);
    colsum(s, 0, (z.L + z.U) * z.H, nullptr, dB1);
    colsum(s, 0, z.H * z.L, nullptr, dB2);
    return after("allegro_layer_backward");
  }
  const SavedLayout sl = saved_layout(z);
  const WorkLayout wl = work_layout(plan, z);
  if ((rc = check_ptr(saved, "saved")) || (rc = check_ptr(workspace, "workspace"))) return rc;
  if (saved_bytes < sl.total)
    return fail(ALLEGRO_E_INVALID, "saved buffer of %zu bytes is smaller than the %zu required", saved_bytes,
                sl.total);
  if (workspace_bytes < wl.total)
    return fail(ALLEGRO_E_INVALID, "workspace of %zu bytes is smaller than the %zu required", workspace_bytes,
                wl.total);
  if (E > 0 && ((rc = check_ptr(h, "h")) || (rc = check_ptr(V, "V")) || (rc = check_ptr(Y, "Y")) ||
                (rc = check_ptr(dh_out, "dh_out")) || (rc = check_ptr(dV_out, "dV_out")) ||
                (rc = check_ptr(dh, "dh")) || (rc = check_ptr(dV, "dV")) || (rc = check_ptr(dY, "dY"))))
    return rc;
  const DenseTable dn = select_dense(L, H);
  const MixTable mx = select_mix(plan->lmax, (plan->flags & ALLEGRO_FULL_PARITY) != 0);
  if (!mx.backward) return fail(ALLEGRO_E_UNSUPPORTED, "no mixing kernel for this plan");
  void *sv_base = const_cast<void *>(saved);
  const float *w = at<float>(sv_base, sl.w), *env = at<float>(sv_base, sl.env), *T = at<float>(sv_base, sl.T);
  const float *sv = at<float>(sv_base, sl.s), *a = at<float>(sv_base, sl.a);
  float *dT = at<float>(workspace, wl.dT), *da = at<float>(workspace, wl.da), *dhm = at<float>(workspace, wl.dhm);
  float *ds = at<float>(workspace, wl.ds), *dw = at<float>(workspace, wl.dw), *genv = at<float>(workspace, wl.genv);
  float *red = at<float>(workspace, wl.red), *mixp = at<float>(workspace, wl.mixp);
  dn.latent_vjp(s, E, h, sv, a, B1, B2, dh_out, da, dhm, ds, red, dB1, dB2);
  mx.backward(s, E, dV_out, T, Mix, ds, dT, mixp, dMix);
  if ((rc = after("allegro_layer_backward"))) return rc;
  if ((rc = allegro_tp_backward_train(plan, N, E, row_ptr, V, env, W, dT, w, Y, dV, genv, dw, dY, dW,
                                      at<void>(workspace, wl.tpws), wl.tpws_bytes, stream)))
    return rc;
  dn.embed_vjp(s, E, h, A, dw, dhm, red, dA, dh);
  return after("allegro_layer_backward");
}

}  // extern "C"
