// MI355X (gfx950) kernels and C ABI of the Allegro channel-wise tensor product.
//
// What is computed is stated in include/allegro_tp.h (arxiv 2504.16068, §II.D:
// the tensor product, its first derivative, and the embedding it consumes).
//
// Mapping (wave64; one workgroup of several waves per center atom):
//   * lane <-> channel u.  With U < 64 a wave holds 64/U lane groups that take
//     interleaved edges of the segment; with U = 128 the workgroup's waves are
//     split between the two channel halves.
//   * The center's slabs (64 consecutive [U][d1] rows, contiguous in HBM) are
//     dealt to its waves; each slab moves through an LDS tile with 16-byte
//     coalesced accesses and each lane then works on its own row.
//   * Direct kernels (forward at lmax <= 2, inference backward at every
//     lmax, training backward at lmax <= 2): path weights W[:, u] and
//     env[n, u, :] are loaded once per center into VGPRs and the contraction
//     runs in registers with the coupling coefficients as instruction literals
//     (generated cores, tp_cores.inc).
//   * Per-center matrices at lmax 3: the forward as out = M x with M built
//     once per center, its rows split over 8 waves (generated TPMFwd); the
//     training backward as grad_x = g M and the per-center products
//     G = sum_e g^T x on the matrix cores (tp_mfma_bwd_kernel, lane tables
//     TPMfmaTab), then the embedding VJP in a launch of its own.
//   * Segment ownership: a center's workgroup owns its env / grad_env rows, so
//     every segmented reduction is a fixed-order sum (registers, then the
//     waves' parts in LDS in wave order) -- no atomics, bit-identical from run
//     to run.
//   * The embedding VJP (grad_w, grad_Y) runs after grad_env is complete, in
//     batches of 8 edges staged in LDS: grad_w lane-per-channel, grad_Y with 8
//     lanes per edge and an xor butterfly over them.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <type_traits>
#include <vector>

#include "allegro_tp.h"
#include "cg_builder.hpp"
#include "device_common.hpp"
#include "plan.hpp"
#include "generated/tp_cores.inc"

namespace {

using namespace allegro_dev;

constexpr int kWave = 64;

// Row stride (floats) for per-lane rows of n floats written to LDS by the 64
// lanes of a wave at once: odd, so that the lanes' rows start in distinct banks.
constexpr int odd_stride(int n) { return n | 1; }

template <int U>
struct Lanes {
  static_assert(U == 16 || U == 32 || U == 64 || U == 128, "U must be 16, 32, 64 or 128");
  static constexpr int LPE = U < kWave ? U : kWave;  // lanes per edge group
  static constexpr int G = kWave / LPE;              // edge groups per wave
  static constexpr int CPL = U / LPE;                // channels per lane
};

// ----------------------------------------------------------------- vector I/O
// Per-lane contiguous rows of D floats; the row start is 4*D-byte aligned
// relative to a 16-byte aligned base, so the widest aligned access is used.
template <int D>
__device__ __forceinline__ void load_row(const float *__restrict__ p, float (&r)[D]) {
  if constexpr (D % 4 == 0) {
#pragma unroll
    for (int i = 0; i < D / 4; ++i) {
      const float4 v = reinterpret_cast<const float4 *>(p)[i];
      r[4 * i] = v.x; r[4 * i + 1] = v.y; r[4 * i + 2] = v.z; r[4 * i + 3] = v.w;
    }
  } else if constexpr (D % 2 == 0) {
#pragma unroll
    for (int i = 0; i < D / 2; ++i) {
      const float2 v = reinterpret_cast<const float2 *>(p)[i];
      r[2 * i] = v.x; r[2 * i + 1] = v.y;
    }
  } else {
#pragma unroll
    for (int i = 0; i < D; ++i) r[i] = p[i];
  }
}

template <int D>
__device__ __forceinline__ void store_row(float *__restrict__ p, const float (&r)[D]) {
  if constexpr (D % 4 == 0) {
#pragma unroll
    for (int i = 0; i < D / 4; ++i)
      reinterpret_cast<float4 *>(p)[i] = make_float4(r[4 * i], r[4 * i + 1], r[4 * i + 2], r[4 * i + 3]);
  } else if constexpr (D % 2 == 0) {
#pragma unroll
    for (int i = 0; i < D / 2; ++i) reinterpret_cast<float2 *>(p)[i] = make_float2(r[2 * i], r[2 * i + 1]);
  } else {
#pragma unroll
    for (int i = 0; i < D; ++i) p[i] = r[i];
  }
}

// acc + fl(a * b) with two separate roundings (no contraction to FMA).
__device__ __forceinline__ float add_rounded_product(float acc, float a, float b) {
#pragma clang fp contract(off)
  const float prod = a * b;
  return acc + prod;
}

// ------------------------------------------------------------ env embedding
// env[n,u,j] = sum_{e in seg(n)} w[e,u] Y[e,j].  Lane groups take different
// centers (U < 64) so every env value is one lane's ascending-e sum.  The
// loads of B edges are issued together and then accumulated in edge order,
// so the summation order (and the deterministic mode's bits) does not change.
template <int U, int D2, bool DET>
__device__ __forceinline__ void env_accumulate(float (&acc)[Lanes<U>::CPL][D2], const float (&wv)[Lanes<U>::CPL],
                                               const float (&y)[D2]) {
#pragma unroll
  for (int t = 0; t < Lanes<U>::CPL; ++t)
#pragma unroll
    for (int j = 0; j < D2; ++j)
      acc[t][j] = DET ? add_rounded_product(acc[t][j], wv[t], y[j]) : __builtin_fmaf(wv[t], y[j], acc[t][j]);
}

// Waves per workgroup of the embedding: each wave takes its own center (or
// its own G centers when U < 64).  One-wave workgroups left too few waves
// resident per compute unit.
constexpr int kEnvWaves = 4;

template <int U, int D2, bool DET>
__global__ __launch_bounds__(kWave * kEnvWaves) void env_embed_kernel(int64_t N, const int64_t *__restrict__ row_ptr,
                                                                      const float *__restrict__ w,
                                                                      const float *__restrict__ Y,
                                                                      float *__restrict__ env) {
  using L = Lanes<U>;
  constexpr int B = D2 <= 9 ? 8 : 4;  // edges whose loads are in flight together
  constexpr int RF = kWave * L::CPL * D2;  // floats of the wave's env rows
  static_assert(RF % 4 == 0, "whole float4 of env rows per wave");
  __shared__ float4 rows4[kEnvWaves * RF / 4];
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
  const int lane = int(threadIdx.x) % kWave, grp = lane / L::LPE, ul = lane % L::LPE;
  const int64_t unit = int64_t(blockIdx.x) * kEnvWaves + wave;
  // with one group per wave the center (hence e and every Y address) is
  // wave-uniform, so Y rows come through scalar loads
  const int64_t n0 = unit * L::G;  // the wave's first center
  if (n0 >= N) return;
  const int64_t n = n0 + (L::G == 1 ? 0 : grp);
  const bool valid = n < N;
  const int64_t e0 = valid ? row_ptr[n] : 0, e1 = valid ? row_ptr[n + 1] : 0;
  float acc[L::CPL][D2];
#pragma unroll
  for (int t = 0; t < L::CPL; ++t)
#pragma unroll
    for (int j = 0; j < D2; ++j) acc[t][j] = 0.0f;
  int64_t e = e0;
  for (; e + B <= e1; e += B) {
    float wv[B][L::CPL], y[B][D2];
#pragma unroll
    for (int b = 0; b < B; ++b) {
#pragma unroll
      for (int j = 0; j < D2; ++j) y[b][j] = Y[(e + b) * D2 + j];
#pragma unroll
      for (int t = 0; t < L::CPL; ++t) wv[b][t] = w[(e + b) * U + ul + t * kWave];
    }
#pragma unroll
    for (int b = 0; b < B; ++b) env_accumulate<U, D2, DET>(acc, wv[b], y[b]);
  }
  for (; e < e1; ++e) {
    float wv[L::CPL], y[D2];
#pragma unroll
    for (int j = 0; j < D2; ++j) y[j] = Y[e * D2 + j];
#pragma unroll
    for (int t = 0; t < L::CPL; ++t) wv[t] = w[e * U + ul + t * kWave];
    env_accumulate<U, D2, DET>(acc, wv, y);
  }
  // The wave's env rows are one contiguous block (its centers are consecutive;
  // lane l's row of channel group t sits at (l + 64 t) D2): staged in LDS and
  // written as 16 bytes per lane along the block, rather than each lane's
  // row on its own (every store instruction touching 64 partial lines).
  float *rows = reinterpret_cast<float *>(rows4) + wave * RF;
#pragma unroll
  for (int t = 0; t < L::CPL; ++t)
#pragma unroll
    for (int j = 0; j < D2; ++j) rows[(lane + kWave * t) * D2 + j] = acc[t][j];
  lds_sync<1>();
  const int64_t base = n0 * U * D2, total = N * U * D2;  // floats
  float4 *dst = reinterpret_cast<float4 *>(env + base);
#pragma unroll
  for (int i = lane; i < RF / 4; i += kWave)
    if (base + 4 * int64_t(i) < total) dst[i] = rows4[wave * (RF / 4) + i];
}

// -------------------------------------------------------------------- slabs
// A center's per-lane rows are streamed in slabs: 64 consecutive rows of D
// floats that are contiguous in HBM, so every slab moves with fully coalesced
// 16-byte accesses (per-lane 72-byte rows read directly cost about a quarter
// of the bandwidth).  With U >= 64, slab (s, t) holds channels t*64 .. t*64+63
// of edge e0+s; with U < 64 it holds edges e0+s*G .. e0+s*G+G-1, all channels,
// and the last slab of a segment may be partial.  A tile of T slabs is staged
// through LDS, where each lane reads and writes its own row.
template <int D>
struct TileShape {
  static constexpr int SF4 = 16 * D;  // float4 per slab (64 rows of D floats)
  // In LDS, 32-float rows are padded to 36 floats, so that the 16-byte reads
  // of eight consecutive lanes' rows (lane r reads row r) hit distinct banks;
  // unpadded, 128-byte rows put all eight on one bank group.  Other widths
  // are odd multiples of a word or short enough to stay as they are.
  static constexpr int RS = D == 32 ? 36 : D;  // LDS row stride (floats)
  static constexpr int LF4 = 16 * RS;          // LDS float4 per slab
  // LDS position of float4 f of a slab
  static __device__ __forceinline__ int pos(int f) { return D == 32 ? f + (f >> 3) : f; }
};

template <int U>
struct Slabs {
  using L = Lanes<U>;
  static __device__ __forceinline__ int64_t count(int64_t deg) { return U >= kWave ? deg : (deg + L::G - 1) / L::G; }
  static __device__ __forceinline__ int64_t first_edge(int64_t e0, int64_t s) {
    return U >= kWave ? e0 + s : e0 + s * L::G;
  }
};

// A tile is cnt consecutive slabs that are also contiguous in memory: any
// number of slabs when U <= 64, one slab when U > 64 (channel halves of
// consecutive edges are U*D floats apart).  Returns the tile's first float4
// (wave-uniform) and how many of its float4 lie inside the segment.
template <int U, int D>
__device__ __forceinline__ int64_t tile_base(int64_t e0, int64_t e1, int64_t s0, int cnt, int t, int &n_f4) {
  constexpr int SF4 = TileShape<D>::SF4;
  if constexpr (U <= kWave) {
    const int64_t eb = Slabs<U>::first_edge(e0, s0);
    const int64_t in_seg = (e1 - eb) * (U * D / 4);
    n_f4 = int(in_seg < int64_t(cnt) * SF4 ? in_seg : int64_t(cnt) * SF4);
    return eb * (U * D / 4);
  } else {
    n_f4 = SF4;  // cnt == 1
    return ((e0 + s0) * U + t * kWave) * D / 4;  // U*D and 64*D are multiples of 4
  }
}

// Cooperative tile moves by the 64 lanes of a wave; TF4 is the float4 count of
// a full tile.  Full tiles take a path without
// per-element predicates: predicated accesses split into basic blocks at which
// the compiler waits for every outstanding memory operation.
template <int U, int D, int TF4>
__device__ __forceinline__ void tile_load(const float *__restrict__ src, float4 *tile, int64_t e0, int64_t e1,
                                          int64_t s0, int cnt, int t, int lane) {
  constexpr int KF = TF4 / kWave, PER = (TF4 + kWave - 1) / kWave;
  int n_f4;
  const float4 *base = reinterpret_cast<const float4 *>(src) + tile_base<U, D>(e0, e1, s0, cnt, t, n_f4);
  float4 v[PER];
  if (n_f4 == TF4) {
#pragma unroll
    for (int k = 0; k < KF; ++k) v[k] = load_stream(base + lane + kWave * k);
    if constexpr (PER > KF) {
      if (lane + kWave * KF < TF4) v[KF] = load_stream(base + lane + kWave * KF);
    }
#pragma unroll
    for (int k = 0; k < KF; ++k) tile[TileShape<D>::pos(lane + kWave * k)] = v[k];
    if constexpr (PER > KF) {
      if (lane + kWave * KF < TF4) tile[TileShape<D>::pos(lane + kWave * KF)] = v[KF];
    }
  } else {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int f = lane + kWave * k;
      v[k] = f < n_f4 ? load_stream(base + f) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int f = lane + kWave * k;
      if (f < n_f4) tile[TileShape<D>::pos(f)] = v[k];
    }
  }
}

template <int U, int D, int TF4>
__device__ __forceinline__ void tile_store(float *__restrict__ dst, const float4 *tile, int64_t e0, int64_t e1,
                                           int64_t s0, int cnt, int t, int lane) {
  constexpr int KF = TF4 / kWave, PER = (TF4 + kWave - 1) / kWave;
  int n_f4;
  float4 *base = reinterpret_cast<float4 *>(dst) + tile_base<U, D>(e0, e1, s0, cnt, t, n_f4);
  if (n_f4 == TF4) {
#pragma unroll
    for (int k = 0; k < KF; ++k) store_stream(tile[TileShape<D>::pos(lane + kWave * k)], base + lane + kWave * k);
    if constexpr (PER > KF) {
      if (lane + kWave * KF < TF4) store_stream(tile[TileShape<D>::pos(lane + kWave * KF)], base + lane + kWave * KF);
    }
  } else {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int f = lane + kWave * k;
      if (f < n_f4) store_stream(tile[TileShape<D>::pos(f)], base + f);
    }
  }
}

// Does lane's row of slab `slab` hold a real edge?  Only partial slabs (U < 64)
// can fail.  For U >= 64 the test is always true, but it is kept as a runtime
// branch: it makes the row contraction its own scheduling region, without
// which the scheduler interleaves it with the tile epilogue and spills.
template <int U>
__device__ __forceinline__ bool row_valid(int64_t e0, int64_t e1, int64_t slab, int lane) {
  if constexpr (U >= kWave) return e0 + slab < e1;
  else return Slabs<U>::first_edge(e0, slab) + lane / U < e1;
}

// ------------------------------------------------------------ path weights
// The lane's weights W[p, u] of its channel u, held in VGPRs.
template <int NP>
struct RegWeights {
  float r[NP];
  __device__ __forceinline__ void load(const float *__restrict__ path_w, int U, int u) {
#pragma unroll
    for (int p = 0; p < NP; ++p) r[p] = path_w[p * U + u];
  }
  __device__ __forceinline__ float operator()(int p) const { return r[p]; }
};

// Path weights read at use from the lane's column of path_w (an L1/L2 hit)
// instead of NP registers, for code run once per center.
struct CachedWeights {
  typedef const __attribute__((address_space(1))) float *gptr;
  gptr col;
  int U;
  __device__ __forceinline__ void load(const float *__restrict__ path_w, int U_, int u) {
    col = (gptr)(path_w + u);
    U = U_;
  }
  __device__ __forceinline__ float operator()(int p) const { return col[p * U]; }
};

template <class Core>
struct KernelTraits {
  // waves per SIMD the register allocation must allow
  static constexpr int kFwdOccupancy = Core::LMAX >= 3 ? 2 : 4;
  static constexpr int kBwdOccupancy = Core::LMAX >= 3 ? 2 : 4;
  static constexpr int bwd_occupancy(bool wg) { return wg ? 2 : kBwdOccupancy; }
};

// Waves per center.  A center's slabs are dealt round robin to NW waves of
// one workgroup (with two channel halves, U = 128, the first NW/2 waves take
// half 0 and the rest half 1); each wave streams its slabs through its own
// LDS tile.  With many waves on one center the concurrently streamed HBM
// regions are few and contiguous: a standalone probe of the forward's access
// pattern measured 4.98 TB/s with one wave per center and 5.51 TB/s with 16.
// That pays where the kernel is HBM-bound (lmax <= 2).  The training backward,
// which also holds the path-weight sums, is bound by VALU issue; with fewer
// waves per center more workgroups fit on a compute unit and overlap one
// center's reduction phases with another's streaming.  The counts are the
// fastest of 1, 2, 4, 8 and 16 measured for each kernel on the MI355X.  (At
// lmax 3 the forward is tp_matrix_kernel and the backward tp_mfma_bwd_kernel.)
template <class Core, int U>
struct TPWaves {
  static constexpr bool kHigh = Core::LMAX >= 3, kWide = U > 64;
  static constexpr int kFwd = 16;  // lmax <= 2
  static constexpr int bwd(bool wg) { return wg ? 4 : (kHigh ? (kWide ? 8 : 4) : 16); }
};

// ------------------------------------------------------ tensor product fwd
template <class Core, int U, int NW = TPWaves<Core, U>::kFwd>
__global__ __launch_bounds__(kWave * NW) __attribute__((amdgpu_waves_per_eu(KernelTraits<Core>::kFwdOccupancy))) void tp_forward_kernel(const int64_t *__restrict__ row_ptr,
                                                           const float *__restrict__ x,
                                                           const float *__restrict__ env,
                                                           const float *__restrict__ path_w,
                                                           float *__restrict__ out) {
  using L = Lanes<U>;
  constexpr int D1 = Core::D1, D2 = Core::D2, WPT = NW / L::CPL;
  constexpr int TF4 = TileShape<D1>::SF4;  // one slab per tile
  static_assert(NW % L::CPL == 0, "waves split evenly over the channel halves");
  __shared__ float4 tiles[NW * TileShape<D1>::LF4];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave, ul = lane % L::LPE;
  const int t = wave / WPT, first = wave % WPT;
  float4 *tile = tiles + wave * TileShape<D1>::LF4;
  float *tile_f = reinterpret_cast<float *>(tile);
  const int64_t n = blockIdx.x;
  const int64_t e0 = row_ptr[n], e1 = row_ptr[n + 1];
  const int64_t n_slabs = Slabs<U>::count(e1 - e0);
  const int u = ul + t * kWave;
  RegWeights<Core::NP> wr;
  wr.load(path_w, U, u);
  float er[D2];
  load_row<D2>(env + (n * U + u) * D2, er);
  for (int64_t s = first; s < n_slabs; s += WPT) {
    tile_load<U, D1, TF4>(x, tile, e0, e1, s, 1, t, lane);
    lds_sync<1>();
    if (row_valid<U>(e0, e1, s, lane)) {
      float *row = tile_f + lane * TileShape<D1>::RS;
      float xr[D1], orow[D1];
#pragma unroll
      for (int i = 0; i < D1; ++i) xr[i] = row[i];
      Core::fwd(xr, er, wr, orow);
#pragma unroll
      for (int i = 0; i < D1; ++i) row[i] = orow[i];
    }
    lds_sync<1>();
    tile_store<U, D1, TF4>(out, tile, e0, e1, s, 1, t, lane);
    lds_sync<1>();
  }
}

// ------------------------------------------ tensor product fwd, lmax 3
// The forward as a per-center matrix (generated TPMFwd): out = M x with
// M[k][i] = sum_{p = (a(i), b, c(k))} W(p) sum_j C_pijk env[j], built once per
// center and channel.  M has about 900 entries per channel at lmax 3, too
// many for one lane, so its rows are split over the NW waves of the center's
// workgroup: every wave reads every row of x and writes ROWS components of
// out.  Tiles of T slabs are staged through LDS rows padded to D1 + 4 floats
// (16-byte row reads by 16 consecutive lanes hit distinct bank quads); every
// thread holds its share of the next tile in registers, so one tile of loads
// is in flight while the current one is computed.  Per edge and channel this
// takes about 900 FMAs instead of about 2,000 instructions, which makes the
// lmax-3 forward HBM-bound.
// s_waitcnt operand that waits until at most n vector memory operations of
// the wave are outstanding (n < 64; lgkmcnt and expcnt left at their maxima):
// the count's low four bits sit at bits 3:0, its high two at bits 15:14.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }

// cache policy bits of a buffer access: non-temporal (streamed once)
constexpr int kNonTemporal = 2;

template <class Core>
constexpr int kMFwdThreads = kWave * TPMFwd<Core::LMAX, Core::FULL>::NW;

// The per-center matrix forward at U = 64 and 128, d1 = 32, with the tiles brought
// into LDS by direct buffer-to-LDS loads instead of through registers: the
// registers the kernel leaves free hold one 32 KB tile, and at one workgroup
// per compute unit one tile in flight leaves HBM latency-bound.  Four tile
// buffers: tile k is multiplied while tiles k + 1 .. k + 3 load (96 KB in
// flight per compute unit; the four buffers and the result tile fill the
// 160 KB of LDS).  A load lands at the LDS address of its lane, so the source
// addresses carry the layout: row r (slab r / 64, channel r % 64) holds its
// 16-byte chunk q at position q ^ s(r), s(r) = (r mod 8) ^ ((r / 8) mod 2), so
// that the rows' 16-byte accesses (lane r reads row r) put any 8 consecutive
// lanes on 8 distinct 16-byte columns and any 16 on distinct bank groups of a
// 256-byte span, without padding (the profiler counts no bank conflicts); the
// result tile uses the same layout.  The waits for a tile's loads are
// explicit (the compiler does not track loads into LDS): every iteration
// issues the same number of loads and stores (past the segment their
// descriptors have no range), so the number issued after tile k's loads is
// fixed.
template <class Core, int U, class MF>
__device__ __forceinline__ void matrix_fwd_dma(const int64_t *__restrict__ row_ptr, const float *__restrict__ x,
                                               const float *__restrict__ env, const float *__restrict__ path_w,
                                               float *__restrict__ out) {
  typedef __attribute__((address_space(3))) void lds_void;
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  using L = Lanes<U>;
  constexpr int D1 = Core::D1, D2 = Core::D2, NW = MF::NW, ROWS = MF::ROWS;
  constexpr int T = 4;                       // slabs per tile (32 KB)
  constexpr int NB = 4;                      // tile buffers
  constexpr int R4 = D1 / 4;                 // float4 per row
  constexpr int TF4 = T * kWave * R4;        // float4 per tile
  constexpr int NT = NW * kWave;
  constexpr int PER = TF4 / NT;              // loads (and stores) per thread and tile
  constexpr uint32_t EDGE_BYTES = U * D1 * 4;
  static_assert(D1 == 32 && U % kWave == 0 && TF4 % NT == 0 && D1 == NW * ROWS && ROWS == 4, "layout");
  // position of 16-byte chunk q of tile row r
  auto pos = [](int r, int q) { return r * R4 + (q ^ ((r & 7) ^ ((r >> 3) & 1))); };
  __shared__ float4 xb4[NB * TF4];
  __shared__ float4 os4[TF4];  // the result tile, laid out as the tile buffers
  const uint32_t xb_lds = uint32_t(reinterpret_cast<uintptr_t>((lds_void *)xb4));
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int64_t n = blockIdx.x;
  const int64_t e0 = row_ptr[n], e1 = row_ptr[n + 1];
  const int64_t n_slabs = e1 - e0;  // one edge per slab (64 channels of one half)
  const int64_t n_tiles = (n_slabs + T - 1) / T;
#pragma unroll 1
  for (int t = 0; t < L::CPL; ++t) {
    const int u = lane + t * kWave;
    // tile k's rows of a [E][U][D1] tensor: a descriptor whose range ends at
    // the segment's last slab (no range past it)
    auto tile_rsrc = [&](const float *base, int64_t k) {
      const int64_t s0 = k * T, cnt = s0 < n_slabs ? (n_slabs - s0 < T ? n_slabs - s0 : T) : 0;
      const float *b = cnt ? base + ((e0 + s0) * U + t * kWave) * D1 : base;
      return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(b), short(0), int(uint32_t(cnt) * EDGE_BYTES),
                                               0x00020000);
    };
    // The loads into LDS are issued from inline assembly so that the
    // compiler's wait insertion, which cannot tell the tile buffers apart,
    // does not make every later LDS access wait for all of them.  LDS address
    // of lane i: m0 + 16 i.
    auto load_tile = [&](int64_t k) {
      const int64_t s0 = k * T, cnt = s0 < n_slabs ? (n_slabs - s0 < T ? n_slabs - s0 : T) : 0;
      const uint64_t b = cnt ? uint64_t(x + ((e0 + s0) * U + t * kWave) * D1) : uint64_t(x);
      const u32x4 rs = {uint32_t(b), uint32_t(b >> 32) & 0xffffu, uint32_t(cnt) * EDGE_BYTES, 0x00020000u};
      const uint32_t dst = xb_lds + uint32_t(k % NB) * uint32_t(TF4 * 16);
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int blk = wave * PER + i, slot = blk * kWave + lane;
        const int r = slot / R4, q = pos(r, slot % R4) - r * R4;  // the chunk that lands at this slot
        const uint32_t voff = uint32_t(r / kWave) * EDGE_BYTES + uint32_t(r % kWave) * (D1 * 4) + uint32_t(q) * 16;
        asm volatile("buffer_load_dwordx4 %0, %1, 0 offen nt lds"
                     :
                     : "v"(voff), "s"(rs), "{m0}"(__builtin_amdgcn_readfirstlane(dst + uint32_t(blk * kWave * 16)))
                     : "memory");
      }
    };
    float m[MF::MAXM];
    {
      CachedWeights wr;
      wr.load(path_w, U, u);
      float er[D2];
      load_row<D2>(env + (n * U + u) * D2, er);
      MF::build(wave, er, wr, m);
    }
    // the loads above are complete before the tile loads start, so that no
    // wait the compiler places for them covers the tile loads
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
#pragma unroll
    for (int k = 0; k < NB - 1; ++k) load_tile(k);
#pragma unroll 1
    for (int64_t k = 0; k < n_tiles; ++k) {
      // loads and stores issued after tile k's loads, per wave: those of
      // tiles k + 1 .. k + NB - 2 and the stores of the tiles in between
      // (PER of each kind per tile)
      if (k == 0)
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * PER));
      else if (k == 1)
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * PER));
      else if (k == 2)
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(4 * PER));
      else
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(5 * PER));
      lds_sync<NW>();  // every wave's share of tile k is in LDS; tile k - 1's buffer is free
      load_tile(k + NB - 1);
      const float4 *xb = xb4 + int(k % NB) * TF4;
      const int cnt = int(n_slabs - k * T < T ? n_slabs - k * T : T);
#pragma unroll 1
      for (int sl = 0; sl < cnt; ++sl) {
        const int r = sl * kWave + lane;
        float xr[D1], o[ROWS];
#pragma unroll
        for (int q = 0; q < R4; ++q) {
          const float4 a = xb[pos(r, q)];
          xr[4 * q] = a.x; xr[4 * q + 1] = a.y; xr[4 * q + 2] = a.z; xr[4 * q + 3] = a.w;
        }
        MF::apply(wave, xr, m, o);
        os4[pos(r, wave)] = make_float4(o[0], o[1], o[2], o[3]);
      }
      lds_sync<NW>();
      const auto ro = tile_rsrc(out, k);
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int f = tid + NT * i, r = f / R4, c = f % R4;
        const uint32_t voff = uint32_t(r / kWave) * EDGE_BYTES + uint32_t(r % kWave) * (D1 * 4) + uint32_t(c) * 16;
        const float4 v = os4[pos(r, c)];
        __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(v.x), __float_as_uint(v.y),
                                                     __float_as_uint(v.z), __float_as_uint(v.w)},
                                               ro, int(voff), 0, kNonTemporal);
      }
    }
    // the loads of the tiles past the end (no range) before the buffers are
    // reused or the workgroup ends
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    lds_sync<NW>();
  }
}

// MF is the generated matrix TPMFwd (out = M x).
template <class Core, int U, class MF>
__global__ __launch_bounds__(kMFwdThreads<Core>) __attribute__((amdgpu_waves_per_eu(2))) void tp_matrix_kernel(
    const int64_t *__restrict__ row_ptr, const float *__restrict__ x, const float *__restrict__ env,
    const float *__restrict__ path_w, float *__restrict__ out) {
  if constexpr (U % kWave == 0 && Core::D1 == 32) {
    matrix_fwd_dma<Core, U, MF>(row_ptr, x, env, path_w, out);
  } else {
    using L = Lanes<U>;
    constexpr int D1 = Core::D1, D2 = Core::D2, NW = MF::NW, ROWS = MF::ROWS;
    constexpr int T = U > kWave ? 4 : 8;      // slabs per tile (32 or 64 KB; 8 at U = 128 would spill)
    constexpr int RS = D1 + 4;                // padded LDS row stride (floats)
    constexpr int R4 = D1 / 4;                // float4 per row
    constexpr int SF4 = TileShape<D1>::SF4;   // float4 per slab
    constexpr int TF4 = T * SF4;              // float4 per tile
    constexpr int NT = NW * kWave;
    constexpr int PER = (TF4 + NT - 1) / NT;  // float4 per thread and tile
    static_assert(D1 % 4 == 0 && D1 == NW * ROWS, "rows of whole float4, split evenly over the waves");
    __shared__ float4 xs4[T * kWave * RS / 4], os4[T * kWave * RS / 4];
    float *xs = reinterpret_cast<float *>(xs4), *os = reinterpret_cast<float *>(os4);
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int64_t n = blockIdx.x;
    const int64_t e0 = row_ptr[n], e1 = row_ptr[n + 1];
    const int64_t n_slabs = Slabs<U>::count(e1 - e0);
    // float4 f of a tile starting at slab s0: its HBM index, or -1 past the segment
    auto src = [&](int64_t s0, int f, int t) -> int64_t {
      const int sl = f / SF4, in = f % SF4;
      if (s0 + sl >= n_slabs) return -1;
      if constexpr (U <= kWave) {
        const int64_t base = Slabs<U>::first_edge(e0, s0) * (U * D1 / 4), end = e1 * (U * D1 / 4);
        const int64_t g = base + f;
        return g < end ? g : -1;
      } else {
        return ((e0 + s0 + sl) * U + t * kWave) * D1 / 4 + in;
      }
    };
  #pragma unroll 1
    for (int t = 0; t < L::CPL; ++t) {
      const int u = lane % L::LPE + t * kWave;
      float4 v[PER];
      auto fetch = [&](int64_t s0) {
        const float4 *x4 = reinterpret_cast<const float4 *>(x);
  #pragma unroll
        for (int i = 0; i < PER; ++i) {
          const int f = tid + NT * i;
          const int64_t g = f < TF4 ? src(s0, f, t) : -1;
          v[i] = g >= 0 ? load_stream(x4 + g) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      };
      // M first: its weight loads would otherwise wait behind the tile's loads
      // (one in-order counter covers both)
      float m[MF::MAXM];
      {
        CachedWeights wr;
        wr.load(path_w, U, u);
        float er[D2];
        load_row<D2>(env + (n * U + u) * D2, er);
        MF::build(wave, er, wr, m);
      }
      if (n_slabs > 0) fetch(0);
      for (int64_t s0 = 0; s0 < n_slabs; s0 += T) {
        // the tile from registers into LDS (padded rows), then the next tile's loads
  #pragma unroll
        for (int i = 0; i < PER; ++i) {
          const int f = tid + NT * i;
          if (f < TF4) *reinterpret_cast<float4 *>(xs + (f / R4) * RS + 4 * (f % R4)) = v[i];
        }
        if (s0 + T < n_slabs) fetch(s0 + T);
        lds_sync<NW>();
        const int cnt = int(n_slabs - s0 < T ? n_slabs - s0 : T);
  #pragma unroll 1
        for (int sl = 0; sl < cnt; ++sl) {
          const int r = sl * kWave + lane;
          float xr[D1], o[ROWS];
  #pragma unroll
          for (int q = 0; q < R4; ++q) {
            const float4 a = *reinterpret_cast<const float4 *>(xs + r * RS + 4 * q);
            xr[4 * q] = a.x; xr[4 * q + 1] = a.y; xr[4 * q + 2] = a.z; xr[4 * q + 3] = a.w;
          }
          MF::apply(wave, xr, m, o);
  #pragma unroll
          for (int k = 0; k < ROWS; ++k) os[r * RS + wave * ROWS + k] = o[k];
        }
        lds_sync<NW>();
        float4 *o4 = reinterpret_cast<float4 *>(out);
  #pragma unroll
        for (int i = 0; i < PER; ++i) {
          const int f = tid + NT * i;
          const int64_t g = f < TF4 ? src(s0, f, t) : -1;
          if (g >= 0) store_stream(*reinterpret_cast<const float4 *>(os + (f / R4) * RS + 4 * (f % R4)), o4 + g);
        }
        // the next iteration writes xs (read above, before the barrier) and then os
        // only after its own barrier, by which every thread has read os here
      }
      lds_sync<NW>();  // both tiles are free before the next channel half
    }
  }
}

// ------------------------------------------------- embedding VJP (pass 2)
// LDS layout of grad_env[n] for the embedding VJP: the U rows of D2 floats in
// eight groups of U / 8 channels.  With D2 % 4 == 0 the rows are read 16 bytes
// at a time and each group is padded to a stride of 4 (mod 8) floats, so that
// the eight lane groups of the grad_Y sums (one channel group each) read
// distinct banks; unpadded, all eight hit the same bank quad.  Other row
// lengths (d2 = 9 at lmax 2) keep the plain layout, which measured faster
// there than an odd stride.
template <int U, int D2>
struct GeRows {
  static constexpr int UQ = U / 8, S0 = UQ * D2;
  static constexpr int PAD = D2 % 4 == 0 ? (S0 % 8 == 4 ? 0 : 4) : 0;
  static constexpr int GS = S0 + PAD, FLOATS = 8 * GS;
  static_assert(U % 8 == 0, "eight channel groups");
  static constexpr int idx(int u, int j) { return (u / UQ) * GS + (u % UQ) * D2 + j; }
};

// The embedding's VJP for the edges [e0, e1) of center n, given its complete
// grad_env[n] rows in LDS (ge_l, GeRows layout), in batches of EB edges dealt round
// robin to the NW waves of the center; each wave first stages the batch's w
// and Y rows in its own LDS area (stage, EB * (U + 1 + D2) floats) with one
// round of coalesced loads:
//   grad_w[e,u] = sum_j grad_env[n,u,j] Y[e,j]   lane <-> channel (coalesced stores)
//   grad_Y[e,j] = sum_u grad_env[n,u,j] w[e,u]   lane <-> (edge k, channel eighth q):
//                 each lane sums U/8 channels, then an xor butterfly over the 8
//                 lanes of the edge (operands swapped between partners, so all 8
//                 hold the same bits)
template <int U, int D2, int NW, int EB>
__device__ __forceinline__ void embedding_vjp(const float *ge_l, float *stage, int64_t e0, int64_t e1, int wave,
                                              int lane, const float *__restrict__ w, const float *__restrict__ Y,
                                              float *__restrict__ grad_w, float *__restrict__ grad_Y) {
  using L = Lanes<U>;
  static_assert(EB == 8, "8 lanes per edge in the grad_Y sums");
  constexpr int WROW = U + 1;  // padded w row: per-lane row reads hit distinct banks
  const int grp = lane / L::LPE, ul = lane % L::LPE;
  float *wl = stage;
  float *yl = wl + EB * WROW;
  const float4 *w4 = reinterpret_cast<const float4 *>(w);
  float gel[L::CPL][D2];
#pragma unroll
  for (int c = 0; c < L::CPL; ++c)
#pragma unroll
    for (int j = 0; j < D2; ++j) gel[c][j] = ge_l[GeRows<U, D2>::idx(ul + c * kWave, j)];
  for (int64_t eb = e0 + int64_t(wave) * EB; eb < e1; eb += int64_t(NW) * EB) {
    const int cnt = int(e1 - eb < EB ? e1 - eb : EB);
    lds_sync<1>();  // this wave's previous batch is done with its staged rows
    for (int i4 = lane; i4 < cnt * (U / 4); i4 += kWave) {
      const float4 v = w4[eb * (U / 4) + i4];
      const int r = (4 * i4) / U, c = (4 * i4) % U;
      float *dst = wl + r * WROW + c;
      dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
    }
    for (int i = lane; i < cnt * D2; i += kWave) yl[i] = Y[eb * D2 + i];
    lds_sync<1>();
    for (int k = grp; k < cnt; k += L::G) {
#pragma unroll
      for (int c = 0; c < L::CPL; ++c) {
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < D2; ++j) acc = __builtin_fmaf(gel[c][j], yl[k * D2 + j], acc);
        grad_w[(eb + k) * U + ul + c * kWave] = acc;
      }
    }
    {
      constexpr int UQ = U / 8;  // channels per lane
      const int k = lane / 8, q = lane % 8;
      const float *wrow = wl + k * WROW + q * UQ;
      const float *gq = ge_l + q * GeRows<U, D2>::GS;
      float gy[D2];
#pragma unroll
      for (int j = 0; j < D2; ++j) gy[j] = 0.0f;
      if (k < cnt) {
#pragma unroll 4
        for (int uu = 0; uu < UQ; ++uu) {
          const float wv = wrow[uu];
#pragma unroll
          for (int j = 0; j < D2; ++j) gy[j] = __builtin_fmaf(gq[uu * D2 + j], wv, gy[j]);
        }
      }
#pragma unroll
      for (int off = 1; off < 8; off *= 2)
#pragma unroll
        for (int j = 0; j < D2; ++j) gy[j] += __shfl_xor(gy[j], off);
      // the batch's grad_Y rows are contiguous: staged in the (no longer
      // needed) Y rows and stored by consecutive lanes, 256 bytes per
      // instruction, instead of one lane per row
      if (k < cnt && q == 0) {
#pragma unroll
        for (int j = 0; j < D2; ++j) yl[k * D2 + j] = gy[j];
      }
      lds_sync<1>();
      float *gyb = grad_Y + eb * D2;
      for (int i = lane; i < cnt * D2; i += kWave) gyb[i] = yl[i];
    }
  }
}

// The embedding VJP as a launch of its own, one workgroup of NW waves per
// center, after a kernel that wrote grad_env (the lmax-3 backward on the
// matrix cores, whose workgroups each own only 16 channels of a center).
template <int U, int D2, int NW>
__global__ __launch_bounds__(kWave * NW) void embedding_vjp_kernel(const int64_t *__restrict__ row_ptr,
                                                                   const float *__restrict__ grad_env,
                                                                   const float *__restrict__ w,
                                                                   const float *__restrict__ Y,
                                                                   float *__restrict__ grad_w,
                                                                   float *__restrict__ grad_Y) {
  using GR = GeRows<U, D2>;
  constexpr int EB = 8, STAGE = EB * (U + 1 + D2);
  static_assert(D2 % 4 == 0 && GR::GS % 4 == 0, "grad_env rows staged 16 bytes at a time");
  __shared__ float4 smem[(GR::FLOATS + NW * STAGE + 3) / 4];
  float *ge_l = reinterpret_cast<float *>(smem);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int64_t n = blockIdx.x;
  const int64_t e0 = row_ptr[n], e1 = row_ptr[n + 1];
  if (e1 <= e0) return;
  const float4 *src = reinterpret_cast<const float4 *>(grad_env + n * U * D2);
  for (int i = tid; i < U * D2 / 4; i += kWave * NW)
    *reinterpret_cast<float4 *>(ge_l + GR::idx(4 * i / D2, 4 * i % D2)) = src[i];
  lds_sync<NW>();
  embedding_vjp<U, D2, NW, EB>(ge_l, ge_l + GR::FLOATS + wave * STAGE, e0, e1, wave, lane, w, Y, grad_w, grad_Y);
}

// ------------------------------------------------------ tensor product bwd
// Pass 1 of one wave: for its slabs of channel half t, grad_x rows in place in
// its x tile, this lane's grad_env partial sums in ge and, with WG, its
// path-weight gradient sums in sw.
template <class Core, int U, bool WG>
__device__ __forceinline__ void bwd_pass1(const float *__restrict__ x, const float *__restrict__ g,
                                          const float *__restrict__ env, const float *__restrict__ path_w,
                                          float *__restrict__ grad_x, float4 *tile_x, float4 *tile_g, int64_t n,
                                          int64_t e0, int64_t e1, int64_t n_slabs, int64_t first, int64_t step,
                                          int t, int lane, float (&ge)[Core::D2], float (&sw)[Core::NP]) {
  constexpr int D1 = Core::D1, D2 = Core::D2, TF4 = TileShape<D1>::SF4;
  const int u = lane % Lanes<U>::LPE + t * kWave;
  RegWeights<Core::NP> wr;
  wr.load(path_w, U, u);
  float er[D2];
  load_row<D2>(env + (n * U + u) * D2, er);
#pragma unroll
  for (int j = 0; j < D2; ++j) ge[j] = 0.0f;
  float *tx = reinterpret_cast<float *>(tile_x);
  const float *tg = reinterpret_cast<const float *>(tile_g);
  for (int64_t s = first; s < n_slabs; s += step) {
    tile_load<U, D1, TF4>(x, tile_x, e0, e1, s, 1, t, lane);
    tile_load<U, D1, TF4>(g, tile_g, e0, e1, s, 1, t, lane);
    lds_sync<1>();
    if (row_valid<U>(e0, e1, s, lane)) {
      // x row in, grad_x row out, in place in the LDS tile
      float *row = tx + lane * TileShape<D1>::RS;
      const float *grow = tg + lane * TileShape<D1>::RS;
      if constexpr (WG) Core::wgrad(row, er, grow, sw);
      Core::bwd(row, er, wr, grow, row, ge);
    }
    lds_sync<1>();
    tile_store<U, D1, TF4>(grad_x, tile_x, e0, e1, s, 1, t, lane);
    lds_sync<1>();
  }
}

// LDS layout of the backward (floats), reused by its phases:
//   pass 1:    NW pairs of x and g tiles;
//   path-weight partial sums: [NW][64][PC] for a chunk of PC paths (WG only);
//   grad_env:  partial sums [NW][64][D2], then grad_env[n] [U][D2], then each
//              wave's staged w and Y rows of pass 2 [NW][EB][U + 1 + D2].
template <class Core, int U, bool WG, int NW_>
struct BwdLds {
  static constexpr int NW = NW_, D2 = Core::D2, NP = Core::NP;
  static constexpr int TILE_F4 = TileShape<Core::D1>::LF4;  // LDS float4 of one tile
  static constexpr int EB = 8;          // edges per pass-2 batch of one wave (8 lanes per edge)
  static constexpr int WROW = U + 1;    // padded w row: per-lane row reads hit distinct banks
  static constexpr int P1 = NW * 2 * TILE_F4 * 4;
  static constexpr int GS = odd_stride(D2);  // row stride of the grad_env partial sums
  static constexpr int GE_PART = NW * kWave * GS;
  static constexpr int GE_ROW = GeRows<U, D2>::FLOATS;
  static constexpr int STAGE = EB * (WROW + D2);
  static constexpr int P2 = GE_PART + GE_ROW + NW * STAGE;
  static constexpr int PC_FIT = (P1 / (NW * kWave) - 1) | 1;  // odd, and its stride fits in P1
  static constexpr int PC = WG ? (NP < PC_FIT ? NP : PC_FIT) : 1;  // paths per reduction chunk
  static constexpr int PS = odd_stride(PC);                        // their row stride
  static constexpr int SW = WG ? NW * kWave * PS : 0;
  static constexpr int FLOATS = P1 > P2 ? (P1 > SW ? P1 : SW) : (P2 > SW ? P2 : SW);
  static_assert(!WG || PC >= 1, "LDS too small for the path-weight partial sums");
};

// With WG the kernel also writes center n's path-weight gradient, summed over
// its edges, to pw_part[n][p][u] (the first of the two reduction stages).
template <class Core, int U, bool WG, int NW = TPWaves<Core, U>::bwd(WG)>
__global__ __launch_bounds__(kWave * NW) __attribute__((amdgpu_waves_per_eu(KernelTraits<Core>::bwd_occupancy(WG)))) void tp_backward_kernel(
        const int64_t *__restrict__ row_ptr, const float *__restrict__ x, const float *__restrict__ env,
        const float *__restrict__ path_w, const float *__restrict__ g, const float *__restrict__ w,
        const float *__restrict__ Y, float *__restrict__ grad_x, float *__restrict__ grad_env,
        float *__restrict__ grad_w, float *__restrict__ grad_Y, float *__restrict__ pw_part) {
  using L = Lanes<U>;
  using B = BwdLds<Core, U, WG, NW>;
  constexpr int D2 = Core::D2, NP = Core::NP, WPT = NW / L::CPL, NT = NW * kWave;
  static_assert(NW % L::CPL == 0, "waves split evenly over the channel halves");
  __shared__ float4 smem[(B::FLOATS + 3) / 4];
  float *lds = reinterpret_cast<float *>(smem);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave, grp = lane / L::LPE, ul = lane % L::LPE;
  const int t = wave / WPT;
  const int64_t n = blockIdx.x;
  const int64_t e0 = row_ptr[n], e1 = row_ptr[n + 1];
  const int64_t n_slabs = Slabs<U>::count(e1 - e0);

  // Pass 1 (lane <-> channel): grad_x per edge, partial sums per wave in registers.
  float ge[D2], sw[NP];
  if constexpr (WG) {
#pragma unroll
    for (int p = 0; p < NP; ++p) sw[p] = 0.0f;
  }
  float4 *tile_x = smem + wave * 2 * B::TILE_F4, *tile_g = tile_x + B::TILE_F4;
  bwd_pass1<Core, U, WG>(x, g, env, path_w, grad_x, tile_x, tile_g, n, e0, e1, n_slabs, wave % WPT, WPT, t, lane,
                         ge, sw);
  lds_sync<NW>();  // every wave is done with its tiles

  if constexpr (WG) {
    // lane groups hold the same channel: butterfly sums in a fixed order (the
    // two operands of each step are swapped between partner lanes, so every
    // lane of a channel ends with the same bits)
#pragma unroll
    for (int p = 0; p < NP; ++p) {
#pragma unroll
      for (int off = L::LPE; off < kWave; off *= 2) sw[p] += __shfl_xor(sw[p], off);
    }
    // then over the waves of the channel half, in wave order, PC paths at a time
    static_for<0, (NP + B::PC - 1) / B::PC>([&](auto ic) {
      constexpr int p0 = decltype(ic)::value * B::PC, pn = NP - p0 < B::PC ? NP - p0 : B::PC;
      if (grp == 0) {
#pragma unroll
        for (int q = 0; q < pn; ++q) lds[(wave * kWave + ul) * B::PS + q] = sw[p0 + q];
      }
      lds_sync<NW>();
      for (int i = tid; i < U * pn; i += NT) {
        const int q = i / U, uu = i % U, tt = uu / kWave, uw = uu % L::LPE;
        float a = 0.0f;
        for (int k = 0; k < WPT; ++k) a += lds[((tt * WPT + k) * kWave + uw) * B::PS + q];
        pw_part[(n * NP + p0 + q) * U + uu] = a;
      }
      lds_sync<NW>();
    });
  }

  // grad_env: the waves' and lane groups' partial sums, in a fixed order
  float *ge_part = lds, *ge_l = lds + B::GE_PART;
#pragma unroll
  for (int j = 0; j < D2; ++j) ge_part[(wave * kWave + lane) * B::GS + j] = ge[j];
  lds_sync<NW>();
  for (int i = tid; i < U * D2; i += NT) {
    const int uu = i / D2, j = i % D2, tt = uu / kWave, uw = uu % L::LPE;
    float a = 0.0f;
    for (int k = 0; k < WPT; ++k)
      for (int q = 0; q < L::G; ++q) a += ge_part[((tt * WPT + k) * kWave + q * L::LPE + uw) * B::GS + j];
    ge_l[GeRows<U, D2>::idx(uu, j)] = a;
    grad_env[n * U * D2 + i] = a;
  }
  lds_sync<NW>();

  // Pass 2: the embedding's VJP through grad_env
  embedding_vjp<U, D2, NW, B::EB>(ge_l, lds + B::GE_PART + B::GE_ROW + wave * B::STAGE, e0, e1, wave, lane, w, Y,
                                  grad_w, grad_Y);
}

// ------------------------------------- backward at lmax 3 on the matrix cores
// Per center n and channel u the backward at lmax 3 is two small dense
// products (d1 = 32 with full parity, 16 without):
//   grad_x[e][i] = sum_k g[e][k] M[k][i],  M[k][i] = sum_{p=(a(i),b,c(k))} W(p) sum_j C_pijk env[j]
//   G[k][i]      = sum_{e in seg(n)} g[e][k] x[e][i]
// (M is the forward's per-center matrix), and the segment sums follow from G:
//   grad_env[j] = sum_{(k,i)} sum_p W(p) C_pijk G[k][i],
//   grad_W[p]  += sum_{(k,i)} sum_j C_pijk env[j] G[k][i]   (training only).
// Both products run on v_mfma_f32_16x16x4f32.  grad_x is formed transposed,
// grad_x^T = M^T g^T: M is the A operand, the 16 edges of a tile are the
// columns and k the reduction (d1 / 4 steps per 16 rows i), so that each lane
// ends with four consecutive columns of one edge's grad_x row and stores them
// as they are.  For G the edges are the reduction (4 per step) and (k, i) the
// 16 x 16 output tiles.  Lane l = 16 h + c holds, in slot s = (tk * NT + ti) *
// 4 + r, the cell (k, i) = (16 tk + 4 h + r, 16 ti + c) of M; of G it holds the
// cell (2 (4 h + r) + tk, 2 c + ti) when d1 = 32 (its operands are read as
// pairs of adjacent columns) and the same cell as of M otherwise.  The
// generated tables (TPMfmaTab) build M's cells and contract G's cells lane by
// lane from the sparse coupling table; M and G cross between the waves in a
// lane-major spill (MfmaShape::spill), 16 bytes at a time.
//
// Work: the pairs (center n, CPW consecutive channels; CPW = 32 / d1, so that a
// pair's row of one edge is 128 contiguous bytes: one channel with full
// parity, two without) are dealt round robin to the streaming waves of a
// persistent grid of one workgroup per compute unit.  Each of the NW
// streaming waves is paired with a helper wave of its own:
//   * the streaming wave moves its pairs' edges in tiles of 16 edges, DEPTH
//     tiles in flight in registers at any time, the tile being multiplied
//     staged in its LDS area (x and g, XOR-swizzled 16-byte columns, so that
//     the row reads of the grad_x operand and the column reads of the G
//     operands are conflict-free), and runs the matrix-core products;
//   * the helper builds the next pair's M and contracts the previous pair's G
//     (grad_env, and the path-weight sums it adds up over its pairs) from the
//     generated lane tables, while its streaming wave keeps streaming; it also
//     writes the zero grad_env rows of pairs without edges.  The helper's work is mostly LDS reads, and the
//     LDS is what it shares with the streaming waves: so it keeps the terms
//     of M it uses most (the first two of each cell) and its H indices in
//     registers (10-bit indices, three to a word), issues the loads of the
//     next pair's path weights and env row before it contracts the previous
//     pair, and runs at a raised wave priority, since a streaming wave waits
//     whenever its helper falls behind.
// They hand M and G over through two LDS buffers of the pair, each guarded by a
// counter: M_ready / M_taken for M (helper writes pair k's M once the wave has
// taken pair k - 1's), G_written / G_taken for G (the wave writes pair k's G
// once the helper has contracted pair k - 1's).  Every wait is bounded; if one
// ever ran out (it cannot, unless the kernel itself is wrong) every later wait
// of the workgroup returns at once and the kernel runs to its end with wrong
// sums.  The streaming wave has no early exit and issues the same memory
// instructions for every tile: either would make the compiler wait for all of
// its loads in flight at every tile.  There is no barrier between waves after
// the tables are loaded.
// The grid is a multiple of U / CPW streaming waves, so every pair a wave
// visits has the same channels: its path-weight sums stay in its helper's LDS
// and leave as one row at the end (a few rows per channel group in all, where
// per-center rows would be hundreds of MB), summed over the waves by
// pw_reduce_waves_kernel.  Every sum has a fixed order.  The embedding VJP,
// which needs all channels of grad_env[n], is embedding_vjp_kernel, launched
// after this kernel.
constexpr int kMfmaEdges = 16;  // edges per tile

template <bool FULL>
struct MfmaShape {
  using Tab = TPMfmaTab<3, FULL>;
  static constexpr int D1 = Tab::D1, D2 = 16, NT = Tab::NT, S = Tab::S, NP = Tab::NP;
  static constexpr int ROW = 32;                 // floats of a pair's row of one edge (128 bytes)
  static constexpr int CPW = ROW / D1;           // channels per pair
  static constexpr int RF4 = ROW / 4;            // float4 per row
  static constexpr int LR = kWave / RF4;         // rows per 16-byte load instruction
  static constexpr int LJ = kMfmaEdges / LR;     // load instructions per tensor and tile
  static constexpr int TILE = kMfmaEdges * ROW;  // floats of one tensor's tile
  static constexpr int DEPTH = 4;                // tiles in flight per streaming wave
  static constexpr int NW = 8, THREADS = 2 * kWave * NW;  // streaming waves, then their helpers
  static constexpr int MB = CPW * S * kWave;     // floats of a pair's M (or G) in lane layout
  static constexpr int HZ = ((Tab::NZ + 2 > Tab::RZ * kWave ? Tab::NZ + 2 : Tab::RZ * kWave) + 3) / 4 * 4;
  // per streaming wave: tile area, M buffer, G buffer; per helper: Z / H
  // scratch, then its path-weight sums (CPW x RPW x 64)
  static constexpr int PWA = CPW * Tab::RPW * kWave;
  static constexpr int AREA = 2 * TILE + 2 * MB, HAREA = HZ + PWA;
  static_assert(NP <= 2 * kWave && Tab::WORDS % 4 == 0 && RF4 * LR == kWave && CPW * D1 == ROW, "layout");
  static constexpr int LDS_FLOATS = Tab::WORDS + NW * AREA + NW * HAREA;
  // float offset of slot group q (slots 4 q .. 4 q + 3) of lane l in a spill of
  // M or G: lane-major, groups XOR-swizzled by (l / 4) mod (S / 4) so that the
  // 16-byte accesses of eight consecutive lanes hit distinct banks
  static __device__ __forceinline__ int spill(int l, int q) { return l * S + 4 * (q ^ ((l >> 2) & (S / 4 - 1))); }
  // first H-table row of round r
  static constexpr int hrow(int r) {
    int o = 0;
    for (int q = 0; q < r; ++q) o += Tab::HT[q];
    return o;
  }
};

// LDS position of element (row e, column k) of a tile of 32-float rows: the
// 16-byte column k / 4 XOR f(e), f(e) = (e & 7) ^ 4 (e & 1), so that the 16
// rows of a tile read at one logical 16-byte column (the grad_x operand: lane
// c reads row c) hit 16 distinct bank groups, while a row stays one 128-byte
// span (the staging writes, and the G operands' column pairs, 16 lanes to a
// row).
__device__ __forceinline__ int swz32(int e, int k) {
  const int f = (e & 7) ^ ((e & 1) << 2);
  return e * 32 + ((((k >> 2) ^ f)) << 2) + (k & 3);
}

// Buffer accesses of a tile: a descriptor of `bytes` bytes from p (raw, 32-bit
// dwords), non-temporal 16-byte loads and stores at a byte offset; a load past
// the range reads zeros and a store past it is dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), short(0), int(bytes), 0x00020000);
}
__device__ __forceinline__ f32x4 load_tile_f4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, int(off), 0, kNonTemporal));
}
__device__ __forceinline__ void store_tile_f4(__amdgpu_buffer_rsrc_t r, uint32_t off, f32x4 v) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, int(off), 0, kNonTemporal);
}

// Counters of the handover between a streaming wave and its helper (LDS).
struct Handover {
  int m_ready, m_taken, g_written, g_taken;
};
constexpr int kSpinLimit = 1 << 24;  // polls before a wait gives up (about a second)
constexpr int kHandoverTimeout = 2;  // bit of the plan's device status word: a handover wait ran out

// Where a handover wait gives up and reports it: after `limit` polls; `status`
// (a device word, or null) gets kHandoverTimeout.
struct WaitCfg {
  int limit;
  int *status;
};

// Waits until *c >= v (acquire); false if the workgroup has stopped or the wait
// ran out, in which case the workgroup is stopped and the timeout reported.
__device__ __forceinline__ bool wait_for(int *c, int v, int *stop, WaitCfg cfg) {
  for (int n = 0; n < cfg.limit; ++n) {
    if (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) >= v) return true;
    if (__hip_atomic_load(stop, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) return false;
    __builtin_amdgcn_s_sleep(1);
  }
  __hip_atomic_store(stop, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  if (cfg.status) __hip_atomic_fetch_or(cfg.status, kHandoverTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return false;
}
__device__ __forceinline__ void post(int *c, int v) {
  __hip_atomic_store(c, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// The pair sequence of one streaming wave (and of its helper): pairs fq,
// fq + total, ... below `pairs`; next() moves to the next pair with edges and
// calls on_empty(n, u0) for each pair it skips.  Everything about it is
// wave-uniform; saying so keeps the tile addresses a scalar base plus 32-bit
// lane offsets.
template <int GROUPS, int CPW>
struct PairWalk {
  int64_t fq, total, pairs, n = 0, eb = 0, e1 = 0;
  int u0 = 0;
  static __device__ __forceinline__ int64_t uniform(int64_t v) {
    const uint64_t u = uint64_t(v);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(u)), hi = __builtin_amdgcn_readfirstlane(uint32_t(u >> 32));
    return int64_t((uint64_t(hi) << 32) | lo);
  }
  template <class F>
  __device__ __forceinline__ bool next(const int64_t *__restrict__ row_ptr, F &&on_empty) {
    while (fq < pairs) {
      n = fq / GROUPS;
      u0 = int(fq % GROUPS) * CPW;
      eb = uniform(row_ptr[n]);
      e1 = uniform(row_ptr[n + 1]);
      fq += total;
      if (e1 > eb) return true;
      on_empty(n, u0);
    }
    return false;
  }
};

template <bool FULL, int U, bool WG>
__global__ __launch_bounds__(MfmaShape<FULL>::THREADS) void tp_mfma_bwd_kernel(
    int64_t N, const int64_t *__restrict__ row_ptr, const float *__restrict__ x, const float *__restrict__ env,
    const float *__restrict__ path_w, const float *__restrict__ g, float *__restrict__ grad_x,
    float *__restrict__ grad_env, float *__restrict__ pw_part, WaitCfg wcfg) {
  using Sh = MfmaShape<FULL>;
  using Tab = typename Sh::Tab;
  constexpr int D1 = Sh::D1, D2 = Sh::D2, NT = Sh::NT, S = Sh::S, NP = Sh::NP, CPW = Sh::CPW;
  constexpr int RF4 = Sh::RF4, LR = Sh::LR, LJ = Sh::LJ, NW = Sh::NW, DEPTH = Sh::DEPTH, GROUPS = U / CPW;
  static_assert(U % CPW == 0, "whole pairs");
  __shared__ float4 smem4[Sh::LDS_FLOATS / 4];
  __shared__ Handover hand[Sh::NW];
  __shared__ int stop;
  float *lds = reinterpret_cast<float *>(smem4);
  const uint32_t *tab = reinterpret_cast<const uint32_t *>(lds);
  const uint16_t *tab16 = reinterpret_cast<const uint16_t *>(lds);
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave), lane = int(threadIdx.x) % kWave;
  const int w = wave % NW;  // the streaming wave of this pair of waves
  float *xs = lds + Tab::WORDS + w * Sh::AREA, *gs = xs + Sh::TILE;
  float *mbuf = gs + Sh::TILE, *gbuf = mbuf + Sh::MB;
  Handover &hv = hand[w];
  {
    const uint4 *src = reinterpret_cast<const uint4 *>(Tab::words());
    for (int i = int(threadIdx.x); i < Tab::WORDS / 4; i += Sh::THREADS) reinterpret_cast<uint4 *>(lds)[i] = src[i];
    if (threadIdx.x < NW) hand[threadIdx.x] = Handover{-1, -1, -1, -1};
    if (threadIdx.x == 0) stop = 0;
  }
  lds_sync<2 * NW>();  // tables and counters are set (the only barrier of the workgroup)
  const int64_t total = int64_t(gridDim.x) * NW, pairs = N * GROUPS;
  constexpr uint32_t EDGE_BYTES = U * D1 * 4;  // between consecutive edges in HBM
  // A lane's offsets within a tile and table offsets are recomputed from
  // opaque values where used: held through the loop (they do not change) they
  // take registers the tiles in flight need.
  auto opaque_lane = [&]() {
    int l = lane;
    __asm__ volatile("" : "+v"(l));
    return l;
  };
  auto opaque_zero = []() {
    int z = 0;
    __asm__ volatile("" : "+s"(z));
    return z;
  };
  PairWalk<GROUPS, CPW> walk{int64_t(blockIdx.x) * NW + w, total, pairs};

  if (wave >= NW) {
    // ------------------------------------------------------------ helper wave
    __builtin_amdgcn_s_setprio(2);
    float *Hz = lds + Tab::WORDS + NW * Sh::AREA + w * Sh::HAREA;
    // path weights and env rows of a pair (lanes 0..67 and 0..15), in three
    // sets: the pair whose M is built (pw0, pw1, pev), the pair whose G is
    // contracted (qw0, qw1, qev) and the next pair, loaded early (nw0, nw1, nev)
    float pw0[CPW], pw1[CPW], pev[CPW], qw0[CPW], qw1[CPW], qev[CPW], nw0[CPW], nw1[CPW], nev[CPW];
    auto load_params = [&](int64_t n, int u0) {
#pragma unroll
      for (int cw = 0; cw < CPW; ++cw) {
        const int u = u0 + cw;
        nw0[cw] = lane < NP ? path_w[lane * U + u] : 0.0f;
        nw1[cw] = lane + kWave < NP ? path_w[(lane + kWave) * U + u] : 0.0f;
        nev[cw] = lane < D2 ? env[(n * U + u) * D2 + lane] : 0.0f;
      }
    };
    auto wp = [&](int cw, int p) {
      const float a = __shfl(pw0[cw], p & 63), b = __shfl(pw1[cw], p & 63);
      return p < kWave ? a : b;
    };
    auto wq = [&](int cw, int p) {
      const float a = __shfl(qw0[cw], p & 63), b = __shfl(qw1[cw], p & 63);
      return p < kWave ? a : b;
    };
    // the lane's M terms 0 and 1 of every slot in registers (coefficients, and
    // Z indices 10 bits each, three to a word); a third term is read from LDS
    static_assert(Tab::NZ + 2 <= 1024 && S * kWave <= 1024, "10-bit table indices");
    constexpr int MTS = (Tab::MT < 2 ? Tab::MT : 2) * S;
    float mc[MTS];
    uint32_t mi[(MTS + 2) / 3];  // three 10-bit indices per word
#pragma unroll
    for (int q = 0; q < MTS; ++q) mc[q] = __uint_as_float(tab[Tab::OFF_MC + q * kWave + lane]);
#pragma unroll
    for (int q = 0; q < (MTS + 2) / 3; ++q) {
      uint32_t v = 0;
#pragma unroll
      for (int b = 0; b < 3; ++b)
        if (3 * q + b < MTS) v |= uint32_t(tab16[2 * Tab::OFF_MI + (3 * q + b) * kWave + lane]) << (10 * b);
      mi[q] = v;
    }
    // the lane's H term indices (10 bits, three per word)
    uint32_t hi[(Tab::TH + 2) / 3];
#pragma unroll
    for (int q = 0; q < (Tab::TH + 2) / 3; ++q) {
      uint32_t v = 0;
#pragma unroll
      for (int b = 0; b < 3; ++b)
        if (3 * q + b < Tab::TH) v |= uint32_t(tab16[2 * Tab::OFF_HI + (3 * q + b) * kWave + lane]) << (10 * b);
      hi[q] = v;
    }
    // M of the pair into the M buffer (the spill layout, per channel of the pair)
    auto build_m = [&]() {
#pragma unroll
      for (int cw = 0; cw < CPW; ++cw) {
        lds_sync<1>();  // Hz is free
#pragma unroll
        for (int r = 0; r < Tab::RZ; ++r) {
          const uint32_t pj = tab[Tab::OFF_ZP + kWave * r + lane];
          Hz[kWave * r + lane] = wp(cw, int(pj & 0xffffu)) * __shfl(pev[cw], int(pj >> 16));
        }
        lds_sync<1>();
#pragma unroll
        for (int sg = 0; sg < S / 4; ++sg) {
          f32x4 a4;
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            const int sl = 4 * sg + r4;
            float a = 0.0f;
#pragma unroll
            for (int t = 0; t < Tab::MT; ++t) {
              const int q = t * S + sl;
              if (q < MTS) {
                a = __builtin_fmaf(mc[q], Hz[(mi[q / 3] >> (10 * (q % 3))) & 0x3ffu], a);
              } else {
                const int row = opaque_zero() + q * kWave + lane;
                a = __builtin_fmaf(__uint_as_float(tab[Tab::OFF_MC + row]), Hz[tab16[2 * Tab::OFF_MI + row]], a);
              }
            }
            a4[r4] = a;
          }
          *reinterpret_cast<f32x4 *>(mbuf + cw * S * kWave + Sh::spill(opaque_lane(), sg)) = a4;
        }
      }
    };
    // The wave's path-weight gradient sums over its pairs, in pair order.  The
    // grid holds a multiple of U / CPW streaming waves, so that a wave's pairs
    // (every total-th) share one channel group; each wave writes one row of
    // CPW x n_paths sums at the end, and a fixed-order sum over the waves of a
    // channel group gives grad_path_w.
    // The sums live in LDS (lane-owned entries, no barrier needed).
    float *pwa = Hz + Sh::HZ;
    auto pwa_at = [&](int cw, int r) -> float & { return pwa[(cw * Tab::RPW + r) * kWave + lane]; };
    if constexpr (WG) {
#pragma unroll
      for (int cw = 0; cw < CPW; ++cw)
#pragma unroll
        for (int r = 0; r < Tab::RPW; ++r) pwa_at(cw, r) = 0.0f;
    }
    auto put_pw = [&]() {
      if constexpr (WG) {
        const int64_t row = (int64_t(blockIdx.x) * NW + w) * CPW;
#pragma unroll
        for (int cw = 0; cw < CPW; ++cw)
#pragma unroll
          for (int r = 0; r < Tab::RPW; ++r)
            if (kWave * r + lane < NP) pw_part[(row + cw) * NP + kWave * r + lane] = pwa_at(cw, r);
      }
    };
    // contraction of the pair's G (in the G buffer): H, grad_env, path-weight sums
    auto contract_g = [&](int64_t n, int u0) {
#pragma unroll
      for (int cw = 0; cw < CPW; ++cw) {
        const int z0 = opaque_zero();
        const int u = u0 + cw;
        const float *Gl = gbuf + cw * S * kWave;
        lds_sync<1>();  // Hz is free
        if (lane == 0) Hz[Tab::NZ] = 0.0f;
        static_for<0, Tab::RH>([&](auto rc) {
          constexpr int r = decltype(rc)::value, r0 = Sh::hrow(r);
          float hv = 0.0f;
#pragma unroll
          for (int t = 0; t < Tab::HT[r]; ++t) {
            const int row = z0 + (r0 + t) * kWave + lane;
            const int q = r0 + t;
            hv = __builtin_fmaf(__uint_as_float(tab[Tab::OFF_HC + row]), Gl[(hi[q / 3] >> (10 * (q % 3))) & 0x3ffu], hv);
          }
          Hz[tab16[2 * Tab::OFF_HT + z0 + r * kWave + lane]] = hv;
          __asm__ volatile("" : : : "memory");
        });
        lds_sync<1>();
        float ge = 0.0f;
#pragma unroll
        for (int t = 0; t < Tab::TGE; ++t) {
          const uint32_t wd = tab[Tab::OFF_GE + z0 + t * kWave + lane];
          ge = __builtin_fmaf(Hz[wd & 0xffffu], wq(cw, int(wd >> 16)), ge);
        }
        ge += __shfl_xor(ge, 1);
        ge += __shfl_xor(ge, 2);
        if ((lane & 3) == 0) grad_env[(n * U + u) * D2 + lane / 4] = ge;
        if constexpr (WG) {
#pragma unroll
          for (int r = 0; r < Tab::RPW; ++r) {
            const int p = kWave * r + lane;
            const uint32_t wd = tab[Tab::OFF_PW + z0 + p];
            const int off = int(wd & 0xffffu), len = int(wd >> 16);
            // the shuffle reads env from lanes 0..15, so every lane takes it:
            // the loop runs to the longest path's length, shorter ones add zeros
            float a = 0.0f;
            for (int k = 0; k < Tab::PWMAX; ++k) {
              const bool in = k < len;
              const uint32_t zp = tab[Tab::OFF_ZP + z0 + (in ? off + k : 0)];
              const float e = __shfl(qev[cw], int(zp >> 16));
              a = __builtin_fmaf(in ? Hz[off + k] : 0.0f, e, a);
            }
            pwa_at(cw, r) += a;  // the wave's pairs all have channel u
          }
        }
      }
    };
    // pairs without edges have zero sums: written here, no tiles
    auto on_empty = [&](int64_t n, int u0) {
      if (lane < CPW * D2) grad_env[(n * U + u0) * D2 + lane] = 0.0f;
    };
    int64_t prev_n = 0;
    int prev_u0 = 0;
    int k = 0;
    auto rotate = [&]() {
#pragma unroll
      for (int cw = 0; cw < CPW; ++cw) {
        qw0[cw] = pw0[cw];
        qw1[cw] = pw1[cw];
        qev[cw] = pev[cw];
        pw0[cw] = nw0[cw];
        pw1[cw] = nw1[cw];
        pev[cw] = nev[cw];
      }
    };
    bool have = walk.next(row_ptr, on_empty);
    if (have) load_params(walk.n, walk.u0);
    rotate();
    while (have) {
      const int64_t cn = walk.n;
      const int cu0 = walk.u0;
      if (!wait_for(&hv.m_taken, k - 1, &stop, wcfg)) {  // the wave has taken the previous M
        put_pw();
        return;
      }
      build_m();
      post(&hv.m_ready, k);
      have = walk.next(row_ptr, on_empty);
      if (have) load_params(walk.n, walk.u0);
      if (k > 0) {
        if (!wait_for(&hv.g_written, k - 1, &stop, wcfg)) {
          put_pw();
          return;
        }
        contract_g(prev_n, prev_u0);
        post(&hv.g_taken, k - 1);
      }
      rotate();
      prev_n = cn;
      prev_u0 = cu0;
      ++k;
    }
    if (k > 0 && wait_for(&hv.g_written, k - 1, &stop, wcfg)) {
      contract_g(prev_n, prev_u0);
      post(&hv.g_taken, k - 1);
    }
    put_pw();
    return;
  }

  // -------------------------------------------------------- streaming wave
  const f32x4 *x4 = reinterpret_cast<const f32x4 *>(x), *g4 = reinterpret_cast<const f32x4 *>(g);
  f32x4 *gx4 = reinterpret_cast<f32x4 *>(grad_x);
  auto no_op = [](int64_t, int) {};
  // the fetch cursor: the next tile to load (edges [feb, feb + 16) of the walk's pair)
  bool fvalid = walk.next(row_ptr, no_op), ffirst = true;
  int64_t feb = walk.eb;
  // the ring of tiles in flight: slot d holds a tile and its identity
  f32x4 vx[DEPTH][LJ], vg[DEPTH][LJ];
  int64_t s_eb[DEPTH], s_e1[DEPTH];
  int s_u0[DEPTH];
  bool s_valid[DEPTH], s_first[DEPTH];
  // Every tile, valid or not, issues the same memory instructions (an empty
  // tile's descriptors have no range: its loads read zeros and its stores are
  // dropped), so that on every path the same loads are in flight and each
  // wait for a tile's data waits for that tile's loads only.
  auto fetch = [&](int d) {
    s_valid[d] = fvalid;
    s_u0[d] = walk.u0;
    s_eb[d] = feb;
    s_e1[d] = walk.e1;
    s_first[d] = ffirst;
    ffirst = false;
    // buffer loads from the tile's first row: rows past the segment lie past
    // the descriptor's range and read as zero
    const int64_t base = (feb * U + walk.u0) * (D1 / 4);
    const uint32_t bytes =
        fvalid ? uint32_t(walk.e1 - feb < kMfmaEdges ? walk.e1 - feb : kMfmaEdges) * EDGE_BYTES : 0u;
    const auto rx = tile_rsrc(x4 + base, bytes), rg = tile_rsrc(g4 + base, bytes);
    const int ln = opaque_lane();
    const uint32_t voff = uint32_t(ln / RF4) * EDGE_BYTES + uint32_t(ln % RF4) * 16u;
#pragma unroll
    for (int j = 0; j < LJ; ++j) {
      vx[d][j] = load_tile_f4(rx, voff + uint32_t(LR * j) * EDGE_BYTES);
      vg[d][j] = load_tile_f4(rg, voff + uint32_t(LR * j) * EDGE_BYTES);
    }
    if (fvalid) {
      feb += kMfmaEdges;
      if (feb >= walk.e1) {
        fvalid = walk.next(row_ptr, no_op);
        ffirst = true;
        feb = walk.eb;
      }
    }
  };

  // the pair whose tiles are being multiplied: its M and G
  float m[CPW][S];
  f32x4 Gacc[CPW][NT * NT];
  int k = -1;  // index of that pair in the wave's sequence
  // G of pair k to the helper (after it has contracted pair k - 1's)
  auto hand_g = [&]() {
    wait_for(&hv.g_taken, k - 1, &stop, wcfg);
#pragma unroll
    for (int cw = 0; cw < CPW; ++cw)
#pragma unroll
      for (int t = 0; t < NT * NT; ++t) *reinterpret_cast<f32x4 *>(gbuf + cw * S * kWave + Sh::spill(opaque_lane(), t)) = Gacc[cw][t];
    post(&hv.g_written, k);
  };
  // one tile, from ring slot d: grad_x rows out, G accumulated
  auto tile = [&](int d) {
    if (s_valid[d] && s_first[d]) {
      if (k >= 0) hand_g();
      ++k;
      wait_for(&hv.m_ready, k, &stop, wcfg);
#pragma unroll
      for (int cw = 0; cw < CPW; ++cw) {
#pragma unroll
        for (int sg = 0; sg < S / 4; ++sg) {
          const f32x4 v = *reinterpret_cast<const f32x4 *>(mbuf + cw * S * kWave + Sh::spill(opaque_lane(), sg));
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) m[cw][4 * sg + r4] = v[r4];
        }
#pragma unroll
        for (int t = 0; t < NT * NT; ++t) Gacc[cw][t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      }
      post(&hv.m_taken, k);
    }
    // the slot's identity, read before fetch(d) below refills the slot
    const int64_t teb = s_eb[d], te1 = s_e1[d];
    const int tu0 = s_u0[d];
    const bool tvalid = s_valid[d];
    int ln = opaque_lane();
    {
      const int le = ln / RF4, lc = ln % RF4;
#pragma unroll
      for (int j = 0; j < LJ; ++j) {
        *reinterpret_cast<f32x4 *>(xs + swz32(le + LR * j, 4 * lc)) = vx[d][j];
        *reinterpret_cast<f32x4 *>(gs + swz32(le + LR * j, 4 * lc)) = vg[d][j];
      }
    }
    fetch(d);  // the slot takes the tile DEPTH ahead
    lds_sync<1>();
    const int h = ln / 16, c = ln % 16;
    // rows past the segment lie past the descriptor's range: not written
    const uint32_t obytes = tvalid ? uint32_t(te1 - teb < kMfmaEdges ? te1 - teb : kMfmaEdges) * EDGE_BYTES : 0u;
    const auto ro = tile_rsrc(gx4 + (teb * U + tu0) * (D1 / 4), obytes);
    static_assert(CPW * NT == 2, "a tile's row is two 16-column blocks");
    f32x4 Dout[2];
#pragma unroll
    for (int cw = 0; cw < CPW; ++cw) {
      // G[k][i] += sum_e g[e][k] x[e][i], four edges (4 st + h) per step
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        float gG[NT], xG[NT];
        if constexpr (Tab::GPAIR) {
          // columns 2 c and 2 c + 1 in one read: tile t takes the columns 2 c + t
          const int o = swz32(4 * st + h, 2 * c);
          const float2 gv = *reinterpret_cast<const float2 *>(gs + o), xv = *reinterpret_cast<const float2 *>(xs + o);
          gG[0] = gv.x;
          gG[1] = gv.y;
          xG[0] = xv.x;
          xG[1] = xv.y;
        } else {
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const int o = swz32(4 * st + h, D1 * cw + 16 * t + c);
            gG[t] = gs[o];
            xG[t] = xs[o];
          }
        }
#pragma unroll
        for (int tk = 0; tk < NT; ++tk)
#pragma unroll
          for (int ti = 0; ti < NT; ++ti)
            Gacc[cw][tk * NT + ti] =
                __builtin_amdgcn_mfma_f32_16x16x4f32(gG[tk], xG[ti], Gacc[cw][tk * NT + ti], 0, 0, 0);
      }
      // grad_x^T[i][e] = sum_k M[k][i] g[e][k], with M as the A operand and the g
      // rows of the 16 edges as B, so that lane 16 h + c ends with the four
      // consecutive columns 16 ti + 4 h .. + 3 of edge c's grad_x row; formed
      // after G, so that its accumulators are not live beside G's operands
      f32x4 gA[NT];
#pragma unroll
      for (int tk = 0; tk < NT; ++tk)
        gA[tk] = *reinterpret_cast<const f32x4 *>(gs + swz32(c, D1 * cw + 16 * tk + 4 * h));
#pragma unroll
      for (int ti = 0; ti < NT; ++ti) {
        f32x4 D = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int tk = 0; tk < NT; ++tk)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            D = __builtin_amdgcn_mfma_f32_16x16x4f32(m[cw][(tk * NT + ti) * 4 + r], gA[tk][r], D, 0, 0, 0);
        Dout[cw * NT + ti] = D;
      }
    }
    // Dout[0] holds columns 4 h .. + 3 of edge c's 32-float row, Dout[1] columns
    // 16 + 4 h .. + 3.  Lanes c and c + 8 trade one of them (a DPP rotation by 8
    // within each row of 16 lanes), so that each store writes eight whole rows
    // of 128 bytes: the first edges c % 8, the second edges c % 8 + 8.
    {
      const bool lo = c < 8;
      const f32x4 snd = lo ? Dout[1] : Dout[0];
      f32x4 rcv;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        rcv[r] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(snd[r]), 0x128, 0xf, 0xf, false));
      const uint32_t col = uint32_t((lo ? 0 : 16) + 4 * h) * 4u, e1 = uint32_t(c & 7);
      store_tile_f4(ro, e1 * EDGE_BYTES + col, lo ? Dout[0] : rcv);
      store_tile_f4(ro, (e1 + 8u) * EDGE_BYTES + col, lo ? rcv : Dout[1]);
    }
    lds_sync<1>();  // the tile's LDS reads are done: the area is free again
  };

#pragma unroll
  for (int d = 0; d < DEPTH; ++d) fetch(d);
  // rounds of DEPTH tiles while any is valid; the empty ones at the end of the
  // sequence run as zero tiles (their products add zeros, their stores drop)
  for (;;) {
    bool any = false;
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) any |= s_valid[d];
    if (!any) break;
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) tile(d);
  }
  if (k >= 0) hand_g();
}

// ------------------------------------------------------ spherical harmonics
// Real harmonics of an edge vector r, component normalisation, as Cartesian
// polynomials of the unit vector u = r/|r| (l <= 3), evaluated in fp64 with
// forward-mode dual numbers so that the same code yields dY/dr exactly.
struct Dual {
  double v, g[3];  // value and gradient with respect to r
};

__device__ __forceinline__ Dual dmul(const Dual &a, const Dual &b) {
  return {a.v * b.v, {a.v * b.g[0] + a.g[0] * b.v, a.v * b.g[1] + a.g[1] * b.v, a.v * b.g[2] + a.g[2] * b.v}};
}
__device__ __forceinline__ Dual dscale(double c, const Dual &a) { return {c * a.v, {c * a.g[0], c * a.g[1], c * a.g[2]}}; }
__device__ __forceinline__ Dual dsub(const Dual &a, const Dual &b) {
  return {a.v - b.v, {a.g[0] - b.g[0], a.g[1] - b.g[1], a.g[2] - b.g[2]}};
}
__device__ __forceinline__ Dual dconst(double c) { return {c, {0.0, 0.0, 0.0}}; }

// Y[0 .. (LMAX+1)^2) of the vector (rx, ry, rz).
template <int LMAX>
__device__ __forceinline__ void real_sh(double rx, double ry, double rz, Dual (&Yd)[(LMAX + 1) * (LMAX + 1)]) {
  const double n2 = rx * rx + ry * ry + rz * rz;
  const double inv = 1.0 / sqrt(n2);  // d(1/|r|)/dr = -r / |r|^3
  const double inv3 = inv * inv * inv;
  const Dual s = {inv, {-rx * inv3, -ry * inv3, -rz * inv3}};
  const Dual x = dmul({rx, {1.0, 0.0, 0.0}}, s), y = dmul({ry, {0.0, 1.0, 0.0}}, s), z = dmul({rz, {0.0, 0.0, 1.0}}, s);
  Yd[0] = dconst(1.0);
  if constexpr (LMAX >= 1) {
    const double c1 = sqrt(3.0);
    Yd[1] = dscale(c1, y);
    Yd[2] = dscale(c1, z);
    Yd[3] = dscale(c1, x);
  }
  if constexpr (LMAX >= 2) {
    const double c15 = sqrt(15.0), c5 = sqrt(5.0);
    const Dual xx = dmul(x, x), yy = dmul(y, y), zz = dmul(z, z);
    Yd[4] = dscale(c15, dmul(x, y));
    Yd[5] = dscale(c15, dmul(y, z));
    Yd[6] = dscale(0.5 * c5, dsub(dscale(3.0, zz), dconst(1.0)));
    Yd[7] = dscale(c15, dmul(x, z));
    Yd[8] = dscale(0.5 * c15, dsub(xx, yy));
    if constexpr (LMAX >= 3) {
      const double a = sqrt(70.0) / 4.0, b = sqrt(105.0), c = sqrt(42.0) / 4.0, d = sqrt(7.0) / 2.0;
      const Dual z5m1 = dsub(dscale(5.0, zz), dconst(1.0));
      Yd[9] = dscale(a, dmul(y, dsub(dscale(3.0, xx), yy)));
      Yd[10] = dscale(b, dmul(dmul(x, y), z));
      Yd[11] = dscale(c, dmul(y, z5m1));
      Yd[12] = dscale(d, dmul(z, dsub(dscale(5.0, zz), dconst(3.0))));
      Yd[13] = dscale(c, dmul(x, z5m1));
      Yd[14] = dscale(0.5 * b, dmul(z, dsub(xx, yy)));
      Yd[15] = dscale(a, dmul(x, dsub(xx, dscale(3.0, yy))));
    }
  }
}

template <int LMAX>
__global__ __launch_bounds__(256) void sh_forward_kernel(int64_t E, const double *__restrict__ vec,
                                                         float *__restrict__ Y) {
  constexpr int D2 = (LMAX + 1) * (LMAX + 1);
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= E) return;
  Dual Yd[D2];
  real_sh<LMAX>(vec[3 * e], vec[3 * e + 1], vec[3 * e + 2], Yd);
#pragma unroll
  for (int j = 0; j < D2; ++j) Y[e * D2 + j] = float(Yd[j].v);
}

template <int LMAX>
__global__ __launch_bounds__(256) void sh_backward_kernel(int64_t E, const double *__restrict__ vec,
                                                          const float *__restrict__ grad_Y,
                                                          double *__restrict__ grad_vec) {
  constexpr int D2 = (LMAX + 1) * (LMAX + 1);
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= E) return;
  Dual Yd[D2];
  real_sh<LMAX>(vec[3 * e], vec[3 * e + 1], vec[3 * e + 2], Yd);
  double gr[3] = {0.0, 0.0, 0.0};
#pragma unroll
  for (int j = 0; j < D2; ++j) {
    const double gy = double(grad_Y[e * D2 + j]);
#pragma unroll
    for (int k = 0; k < 3; ++k) gr[k] += gy * Yd[j].g[k];
  }
#pragma unroll
  for (int k = 0; k < 3; ++k) grad_vec[3 * e + k] = gr[k];
}

// ------------------------------------------------------------- CSR check
__global__ void zero_word_kernel(int *word) { *word = 0; }

__global__ void csr_check_kernel(int64_t N, int64_t E, const int64_t *__restrict__ row_ptr, int *status) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i <= N; i += stride) {
    const int64_t v = row_ptr[i];
    bool bad = v < 0 || v > E;
    if (i == 0 && v != 0) bad = true;
    if (i == N && v != E) bad = true;
    if (i < N && row_ptr[i + 1] < v) bad = true;
    if (bad) atomicOr(status, 1);
  }
}

// ------------------------------------------- path-weight gradient reduction
// Stages two and three of grad_path_w: column c = p * U + u of pw_part[N][P*U]
// is summed over the centers, first within kPwChunks fixed ranges of rows, then
// over the ranges, each sum in a fixed order (run-to-run bit-identical).
constexpr int kPwChunks = 128;

__global__ __launch_bounds__(256) void pw_reduce_rows_kernel(int64_t N, int cols, const float *__restrict__ part,
                                                             float *__restrict__ chunk_sums) {
  const int c = int(blockIdx.x) * 256 + int(threadIdx.x);
  if (c >= cols) return;
  const int64_t per = (N + kPwChunks - 1) / kPwChunks;
  const int64_t r0 = int64_t(blockIdx.y) * per;
  const int64_t r1 = r0 + per < N ? r0 + per : N;
  float a0 = 0.0f, a1 = 0.0f, a2 = 0.0f, a3 = 0.0f;
  int64_t r = r0;
  for (; r + 4 <= r1; r += 4) {
    a0 += part[r * cols + c];
    a1 += part[(r + 1) * cols + c];
    a2 += part[(r + 2) * cols + c];
    a3 += part[(r + 3) * cols + c];
  }
  for (; r < r1; ++r) a0 += part[r * cols + c];
  chunk_sums[int64_t(blockIdx.y) * cols + c] = (a0 + a1) + (a2 + a3);
}

__global__ __launch_bounds__(256) void pw_reduce_chunks_kernel(int rows, int cols, const float *__restrict__ chunk_sums,
                                                               float *__restrict__ grad_pw) {
  const int c = int(blockIdx.x) * 256 + int(threadIdx.x);
  if (c >= cols) return;
  float a = 0.0f;
  for (int r = 0; r < rows; ++r) a += chunk_sums[int64_t(r) * cols + c];
  grad_pw[c] = a;
}

// The matrix-core backward's path-weight rows: part[R][U][np], one row per
// streaming wave; grad_pw[p][u] is the sum over r of part[r][u][p], in order.
__global__ __launch_bounds__(256) void pw_reduce_waves_kernel(int R, int U, int np, const float *__restrict__ part,
                                                              float *__restrict__ grad_pw) {
  const int c = int(blockIdx.x) * 256 + int(threadIdx.x);
  if (c >= U * np) return;
  const int p = c / U, u = c % U;
  float a = 0.0f;
  for (int r = 0; r < R; ++r) a += part[(int64_t(r) * U + u) * np + p];
  grad_pw[c] = a;
}

__global__ __launch_bounds__(256) void zero_floats_kernel(int n, float *__restrict__ p) {
  const int i = int(blockIdx.x) * 256 + int(threadIdx.x);
  if (i < n) p[i] = 0.0f;
}

// ------------------------------------------- allocation-free training backward
// The path-weight partial sums of allegro_tp_backward_train_noalloc live in a
// file-scope device array instead of a caller workspace: kNoAllocFloats fp32
// (64 MiB), held by every GPU the library runs on until the process ends.
constexpr int64_t kNoAllocFloats = int64_t(16) << 20;
constexpr int64_t kNoAllocChunks = 256;  // chunk rows kept for the last sum
constexpr int kMaxPwRounds = 1024;        // per-wave row rounds of the matrix-core backward
static __device__ __align__(256) float scratch[kNoAllocFloats];

// ------------------------------------------------------------- host side
using allegro_internal::fail;

struct NoAllocLayout {
  int64_t centers;  // centers per chunk
};

// rows of cols floats: [centers][cols] per-center sums, [128][cols] range sums,
// [kNoAllocChunks][cols] chunk sums
NoAllocLayout noalloc_layout(int cols) {
  const int64_t rows = kNoAllocFloats / cols;
  return {rows - kPwChunks - kNoAllocChunks};
}

// Device address of `scratch` on the current device, looked up once per device
// (each GPU holds its own copy of the array at its own address).
int noalloc_scratch(float **out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static float *addr[kMaxDevices] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(ALLEGRO_E_HIP, "no current HIP device for the static scratch (device %d)", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    const hipError_t err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess || !p)
      return fail(ALLEGRO_E_HIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev, hipGetErrorString(err));
    addr[dev] = static_cast<float *>(p);
  }
  *out = addr[dev];
  return ALLEGRO_OK;
}

bool misaligned(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

using EnvFn = void (*)(dim3, hipStream_t, int64_t, const int64_t *, const float *, const float *, float *);
using FwdFn = void (*)(dim3, hipStream_t, const int64_t *, const float *, const float *, const float *, float *);
using BwdFn = void (*)(dim3, hipStream_t, const int64_t *, const float *, const float *, const float *, const float *,
                       const float *, const float *, float *, float *, float *, float *, float *, WaitCfg);

template <int U, int D2, bool DET>
void launch_env(dim3 grid, hipStream_t s, int64_t N, const int64_t *rp, const float *w, const float *Y, float *env) {
  hipLaunchKernelGGL((env_embed_kernel<U, D2, DET>), grid, dim3(kWave * kEnvWaves), 0, s, N, rp, w, Y, env);
}

template <class Core, int U>
void launch_fwd(dim3 grid, hipStream_t s, const int64_t *rp, const float *x, const float *env, const float *pw,
                float *out) {
  if constexpr (Core::LMAX >= 3)
    hipLaunchKernelGGL((tp_matrix_kernel<Core, U, TPMFwd<Core::LMAX, Core::FULL>>), grid, dim3(kMFwdThreads<Core>), 0,
                       s, rp, x, env, pw, out);
  else
    hipLaunchKernelGGL((tp_forward_kernel<Core, U>), grid, dim3(kWave * TPWaves<Core, U>::kFwd), 0, s, rp, x, env, pw,
                       out);
}

// Persistent grid of the matrix-core backward: the workgroups resident on the
// device at once (compute units x workgroups per unit), at most one wave per
// pair of work.  Looked up once per device and kernel.
template <bool FULL, int U, bool WG>
unsigned mfma_grid(int64_t N) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static int resident[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = 0;
  int res;
  {
    std::lock_guard<std::mutex> lock(mu);
    if (!resident[dev]) {
      int cus = 0, per = 0;
      if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 256;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, tp_mfma_bwd_kernel<FULL, U, WG>,
                                                       MfmaShape<FULL>::THREADS, 0) != hipSuccess ||
          per < 1)
        per = 1;
      resident[dev] = cus * per;
    }
    res = resident[dev];
  }
  // a multiple of GB workgroups, so that the streaming waves number a
  // multiple of the channel groups (each wave keeps one group)
  constexpr int GROUPS = U / MfmaShape<FULL>::CPW, GB = GROUPS / MfmaShape<FULL>::NW;
  static_assert(GROUPS % MfmaShape<FULL>::NW == 0, "whole channel groups per round of waves");
  const int64_t blocks = N * GB;  // one streaming wave per pair
  int64_t cap = res >= GB ? res / GB * GB : GB;
  if (cap > int64_t(kMaxPwRounds) * GB) cap = int64_t(kMaxPwRounds) * GB;
  return unsigned(blocks < cap ? blocks : cap);
}

// Rows of U x n_paths path-weight sums the matrix-core backward writes for N
// centers: one per round of streaming waves over the channel groups, at most
// min(N, kMaxPwRounds) on any device.
template <bool FULL, int U>
int64_t mfma_pw_rounds(int64_t N) {
  return int64_t(mfma_grid<FULL, U, true>(N)) * MfmaShape<FULL>::NW / (U / MfmaShape<FULL>::CPW);
}

template <class Core, int U, bool WG>
void launch_bwd(dim3 grid, hipStream_t s, const int64_t *rp, const float *x, const float *env, const float *pw,
                const float *g, const float *w, const float *Y, float *gx, float *genv, float *gw, float *gy,
                float *pw_part, WaitCfg wcfg) {
  if constexpr (Core::LMAX >= 3 && WG) {
    // training backward at lmax 3: grad_x, grad_env and per-wave path-weight
    // sums on the matrix cores (one read of x and g), then the embedding VJP from the
    // complete grad_env.  The inference backward stays on the direct kernel,
    // which is faster there (10.3 against 12.0 ms on 20,000 centers, U = 128).
    const int64_t N = grid.x;
    hipLaunchKernelGGL((tp_mfma_bwd_kernel<Core::FULL, U, WG>), dim3(mfma_grid<Core::FULL, U, WG>(N)),
                       dim3(MfmaShape<Core::FULL>::THREADS), 0, s, N, rp, x, env, pw, g, gx, genv, pw_part, wcfg);
    hipLaunchKernelGGL((embedding_vjp_kernel<U, Core::D2, 4>), grid, dim3(kWave * 4), 0, s, rp, genv, w, Y, gw, gy);
  } else {
    hipLaunchKernelGGL((tp_backward_kernel<Core, U, WG>), grid, dim3(kWave * TPWaves<Core, U>::bwd(WG)), 0, s, rp, x,
                       env, pw, g, w, Y, gx, genv, gw, gy, pw_part);
  }
}

struct Kernels {
  EnvFn env = nullptr;
  FwdFn fwd = nullptr;
  BwdFn bwd = nullptr;
  BwdFn bwd_wg = nullptr;  // also writes path-weight gradient partial sums
  // matrix-core training backward: rounds of per-wave path-weight rows it
  // writes for N centers (null for the direct kernels' per-center rows)
  int64_t (*pw_rounds)(int64_t N) = nullptr;
};

template <int LMAX, bool FULL, int U>
Kernels kernels_for(bool det) {
  using Core = TPCore<LMAX, FULL>;
  Kernels k;
  k.env = det ? &launch_env<U, Core::D2, true> : &launch_env<U, Core::D2, false>;
  k.fwd = &launch_fwd<Core, U>;
  k.bwd = &launch_bwd<Core, U, false>;
  k.bwd_wg = &launch_bwd<Core, U, true>;
  if constexpr (LMAX >= 3) k.pw_rounds = &mfma_pw_rounds<FULL, U>;
  return k;
}

template <int LMAX, bool FULL>
Kernels kernels_for_u(int U, bool det) {
  switch (U) {
    case 16: return kernels_for<LMAX, FULL, 16>(det);
    case 32: return kernels_for<LMAX, FULL, 32>(det);
    case 64: return kernels_for<LMAX, FULL, 64>(det);
    case 128: return kernels_for<LMAX, FULL, 128>(det);
    default: return {};
  }
}

Kernels select(const allegro_tp_plan *p) {
  const bool full = (p->flags & ALLEGRO_FULL_PARITY) != 0, det = (p->flags & ALLEGRO_DETERMINISTIC) != 0;
  switch (p->lmax * 2 + (full ? 1 : 0)) {
    case 2: return kernels_for_u<1, false>(p->U, det);
    case 3: return kernels_for_u<1, true>(p->U, det);
    case 4: return kernels_for_u<2, false>(p->U, det);
    case 5: return kernels_for_u<2, true>(p->U, det);
    case 6: return kernels_for_u<3, false>(p->U, det);
    case 7: return kernels_for_u<3, true>(p->U, det);
    default: return {};
  }
}

int check_sizes(const allegro_tp_plan *p, int64_t N, int64_t E, const int64_t *row_ptr) {
  if (!p) return fail(ALLEGRO_E_INVALID, "plan is NULL");
  if (N < 0 || E < 0) return fail(ALLEGRO_E_INVALID, "negative size (N=%lld, E=%lld)", (long long)N, (long long)E);
  if (N == 0 && E > 0) return fail(ALLEGRO_E_INVALID, "E=%lld edges but N=0 centers", (long long)E);
  if (N >= (int64_t(1) << 31)) return fail(ALLEGRO_E_INVALID, "N=%lld exceeds 2^31-1", (long long)N);
  if (N > 0 && !row_ptr) return fail(ALLEGRO_E_INVALID, "row_ptr is NULL");
  if (row_ptr && (reinterpret_cast<uintptr_t>(row_ptr) & 7u))
    return fail(ALLEGRO_E_INVALID, "row_ptr is not 8-byte aligned");
  return ALLEGRO_OK;
}

int check_tensor(const void *ptr, const char *name) {
  if (!ptr) return fail(ALLEGRO_E_INVALID, "%s is NULL", name);
  if (misaligned(ptr)) return fail(ALLEGRO_E_INVALID, "%s is not 16-byte aligned", name);
  return ALLEGRO_OK;
}

// The device CSR check of ALLEGRO_VALIDATE; the caller holds p->validate_mu.
// On success the status word is zero.
int validate_csr_locked(allegro_tp_plan *p, int64_t N, int64_t E, const int64_t *row_ptr, hipStream_t s) {
  hipLaunchKernelGGL(zero_word_kernel, dim3(1), dim3(1), 0, s, p->status);
  const int64_t blocks = std::min<int64_t>((N + 256) / 256, 4096);
  hipLaunchKernelGGL(csr_check_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, N, E, row_ptr, p->status);
  int host = 0;
  if (hipMemcpyAsync(&host, p->status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(ALLEGRO_E_HIP, "CSR validation failed to run: %s", hipGetErrorString(hipGetLastError()));
  if (host) return fail(ALLEGRO_E_INVALID, "row_ptr is not a valid CSR pointer for N=%lld, E=%lld", (long long)N,
                        (long long)E);
  return ALLEGRO_OK;
}

int validate_csr(allegro_tp_plan *p, int64_t N, int64_t E, const int64_t *row_ptr, hipStream_t s) {
  std::lock_guard<std::mutex> lock(p->validate_mu);
  return validate_csr_locked(p, N, E, row_ptr, s);
}

// After the launches of a validated training backward (p->validate_mu held, the
// status word zeroed by the CSR check): waits for them and reports a handover
// wait of the matrix-core kernel that ran out.
int check_handover_locked(allegro_tp_plan *p, hipStream_t s, const char *what) {
  int host = 0;
  if (hipMemcpyAsync(&host, p->status, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(ALLEGRO_E_HIP, "%s: reading the device status failed: %s", what, hipGetErrorString(hipGetLastError()));
  if (host & kHandoverTimeout)
    return fail(ALLEGRO_E_TIMEOUT, "%s: a wait between the matrix-core kernel's waves ran out; the outputs are not valid",
                what);
  return ALLEGRO_OK;
}

int after_launch(const char *what) {
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(ALLEGRO_E_HIP, "%s launch failed: %s", what, hipGetErrorString(err));
  return ALLEGRO_OK;
}

// Blocks of 64 lanes: the env kernel packs 64/U centers per block when U < 64.
unsigned env_blocks(int U, int64_t N) {
  const int64_t per = (U < kWave ? kWave / U : 1) * int64_t(kEnvWaves);  // centers per workgroup
  return unsigned((N + per - 1) / per);
}

}  // namespace

extern "C" {

// Failure injection for tests: ALLEGRO_SIMULATE_ALLOC_FAILURE = "plan", "table"
// or "status" makes that allocation of plan creation fail as if memory were
// exhausted (the status word's hipMalloc is then not called).
static bool simulated_alloc_failure(const char *what) {
  const char *v = std::getenv("ALLEGRO_SIMULATE_ALLOC_FAILURE");
  return v && std::strcmp(v, what) == 0;
}

// Failure injection for tests: with ALLEGRO_SIMULATE_HANDOVER_TIMEOUT set (to
// anything) at plan creation, every wait between the waves of the matrix-core
// backward gives up at once, as if the partner wave had stalled; the kernel
// still runs to its end, and a validating plan reports ALLEGRO_E_TIMEOUT.
static bool simulated_handover_timeout() { return std::getenv("ALLEGRO_SIMULATE_HANDOVER_TIMEOUT") != nullptr; }

int allegro_tp_plan_create(allegro_tp_plan **plan, int lmax, int U, int flags) {
  if (!plan) return fail(ALLEGRO_E_INVALID, "plan output pointer is NULL");
  *plan = nullptr;
  if (lmax < 1 || lmax > 3) return fail(ALLEGRO_E_UNSUPPORTED, "lmax=%d not supported (1, 2 or 3)", lmax);
  if (U != 16 && U != 32 && U != 64 && U != 128)
    return fail(ALLEGRO_E_UNSUPPORTED, "U=%d not supported (16, 32, 64 or 128)", U);
  if (flags & ~(ALLEGRO_FULL_PARITY | ALLEGRO_DETERMINISTIC | ALLEGRO_VALIDATE))
    return fail(ALLEGRO_E_INVALID, "unknown flags 0x%x", flags);
  allegro_tp_plan *p = simulated_alloc_failure("plan") ? nullptr : new (std::nothrow) allegro_tp_plan;
  if (!p) return fail(ALLEGRO_E_NOMEM, "plan allocation failed");
  p->lmax = lmax;
  p->U = U;
  p->flags = flags;
  if (simulated_handover_timeout()) p->spin_limit = 0;
  try {
    if (simulated_alloc_failure("table")) throw std::bad_alloc();
    p->table = allegro::build_table(lmax, (flags & ALLEGRO_FULL_PARITY) != 0);
  } catch (const std::bad_alloc &) {
    delete p;
    return fail(ALLEGRO_E_NOMEM, "coupling table allocation failed");
  } catch (const std::exception &ex) {
    delete p;
    return fail(ALLEGRO_E_INVALID, "coupling table build failed: %s", ex.what());
  }
  if (flags & ALLEGRO_VALIDATE) {
    if (simulated_alloc_failure("status")) {
      delete p;
      return fail(ALLEGRO_E_NOMEM, "device status word allocation failed (simulated)");
    }
    if (hipMalloc(&p->status, sizeof(int)) != hipSuccess) {
      p->status = nullptr;
      delete p;
      return fail(ALLEGRO_E_NOMEM, "device status word allocation failed: %s", hipGetErrorString(hipGetLastError()));
    }
  }
  *plan = p;
  return ALLEGRO_OK;
}

int allegro_tp_plan_destroy(allegro_tp_plan *plan) {
  if (!plan) return ALLEGRO_OK;
  if (plan->status) (void)hipFree(plan->status);
  delete plan;
  return ALLEGRO_OK;
}

int allegro_tp_plan_query(const allegro_tp_plan *plan, int *d1, int *d2, int *n_paths, int *path_desc, int *nnz) {
  if (!plan) return fail(ALLEGRO_E_INVALID, "plan is NULL");
  const auto &t = plan->table;
  if (d1) *d1 = t.d1;
  if (d2) *d2 = t.d2;
  if (n_paths) *n_paths = int(t.paths.size());
  if (nnz) *nnz = int(t.entries.size());
  if (path_desc)
    for (size_t p = 0; p < t.paths.size(); ++p) {
      const auto &ph = t.paths[p];
      const int row[6] = {t.x_irreps[ph.a].l, t.x_irreps[ph.a].p, t.env_irreps[ph.b].l,
                          t.env_irreps[ph.b].p, t.x_irreps[ph.c].l, t.x_irreps[ph.c].p};
      std::memcpy(path_desc + 6 * p, row, sizeof row);
    }
  return ALLEGRO_OK;
}

int allegro_tp_plan_cg(const allegro_tp_plan *plan, int *idx, double *val) {
  if (!plan) return fail(ALLEGRO_E_INVALID, "plan is NULL");
  if (!idx || !val) return fail(ALLEGRO_E_INVALID, "output array is NULL");
  const auto &es = plan->table.entries;
  for (size_t q = 0; q < es.size(); ++q) {
    idx[4 * q] = es[q].path;
    idx[4 * q + 1] = es[q].i;
    idx[4 * q + 2] = es[q].j;
    idx[4 * q + 3] = es[q].k;
    val[q] = es[q].value;
  }
  return ALLEGRO_OK;
}

int allegro_env_embed(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr, const float *w,
                      const float *Y, float *env, void *stream) {
  int rc = check_sizes(plan, N, E, row_ptr);
  if (rc) return rc;
  if (N == 0) return ALLEGRO_OK;
  if ((rc = check_tensor(env, "env"))) return rc;
  if (E > 0 && ((rc = check_tensor(w, "w")) || (rc = check_tensor(Y, "Y")))) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto *mp = const_cast<allegro_tp_plan *>(plan);
  if ((plan->flags & ALLEGRO_VALIDATE) && (rc = validate_csr(mp, N, E, row_ptr, s))) return rc;
  const Kernels k = select(plan);
  if (!k.env) return fail(ALLEGRO_E_UNSUPPORTED, "no kernel for this plan");
  k.env(dim3(env_blocks(plan->U, N)), s, N, row_ptr, w, Y, env);
  return after_launch("allegro_env_embed");
}

int allegro_tp_forward(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr, const float *x,
                       const float *env, const float *path_w, float *out, void *stream) {
  int rc = check_sizes(plan, N, E, row_ptr);
  if (rc) return rc;
  if (E == 0) return ALLEGRO_OK;
  if ((rc = check_tensor(x, "x")) || (rc = check_tensor(env, "env")) || (rc = check_tensor(path_w, "path_w")) ||
      (rc = check_tensor(out, "out")))
    return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto *mp = const_cast<allegro_tp_plan *>(plan);
  if ((plan->flags & ALLEGRO_VALIDATE) && (rc = validate_csr(mp, N, E, row_ptr, s))) return rc;
  const Kernels k = select(plan);
  if (!k.fwd) return fail(ALLEGRO_E_UNSUPPORTED, "no kernel for this plan");
  k.fwd(dim3(unsigned(N)), s, row_ptr, x, env, path_w, out);
  return after_launch("allegro_tp_forward");
}

int allegro_tp_backward(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr, const float *x,
                        const float *env, const float *path_w, const float *grad_out, const float *w, const float *Y,
                        float *grad_x, float *grad_env, float *grad_w, float *grad_Y, void *stream) {
  int rc = check_sizes(plan, N, E, row_ptr);
  if (rc) return rc;
  if (N == 0) return ALLEGRO_OK;
  if ((rc = check_tensor(grad_env, "grad_env")) || (rc = check_tensor(env, "env")) ||
      (rc = check_tensor(path_w, "path_w")))
    return rc;
  if (E > 0 && ((rc = check_tensor(x, "x")) || (rc = check_tensor(grad_out, "grad_out")) ||
                (rc = check_tensor(w, "w")) || (rc = check_tensor(Y, "Y")) || (rc = check_tensor(grad_x, "grad_x")) ||
                (rc = check_tensor(grad_w, "grad_w")) || (rc = check_tensor(grad_Y, "grad_Y"))))
    return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto *mp = const_cast<allegro_tp_plan *>(plan);
  if ((plan->flags & ALLEGRO_VALIDATE) && (rc = validate_csr(mp, N, E, row_ptr, s))) return rc;
  const Kernels k = select(plan);
  if (!k.bwd) return fail(ALLEGRO_E_UNSUPPORTED, "no kernel for this plan");
  k.bwd(dim3(unsigned(N)), s, row_ptr, x, env, path_w, grad_out, w, Y, grad_x, grad_env, grad_w, grad_Y, nullptr,
        WaitCfg{plan->spin_limit, nullptr});
  return after_launch("allegro_tp_backward");
}

int allegro_tp_backward_workspace(const allegro_tp_plan *plan, int64_t N, size_t *bytes) {
  if (!plan) return fail(ALLEGRO_E_INVALID, "plan is NULL");
  if (N < 0 || N >= (int64_t(1) << 31)) return fail(ALLEGRO_E_INVALID, "N=%lld out of range", (long long)N);
  if (!bytes) return fail(ALLEGRO_E_INVALID, "bytes is NULL");
  const int64_t cols = int64_t(plan->table.paths.size()) * plan->U;
  // the matrix-core kernel's per-wave rows (one per round of its waves over
  // the channel groups: at most one per center and at most kMaxPwRounds; a
  // bound that needs no device query), else one row per center and the range
  // sums
  const int64_t rows = select(plan).pw_rounds ? std::max<int64_t>(std::min<int64_t>(N, kMaxPwRounds), 1)
                                              : N + kPwChunks;
  *bytes = size_t(rows * cols) * sizeof(float);
  return ALLEGRO_OK;
}

int allegro_tp_backward_train(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr,
                              const float *x, const float *env, const float *path_w, const float *grad_out,
                              const float *w, const float *Y, float *grad_x, float *grad_env, float *grad_w,
                              float *grad_Y, float *grad_path_w, void *workspace, size_t workspace_bytes,
                              void *stream) {
  int rc = check_sizes(plan, N, E, row_ptr);
  if (rc) return rc;
  if ((rc = check_tensor(grad_path_w, "grad_path_w"))) return rc;
  const int cols = int(plan->table.paths.size()) * plan->U;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (N == 0) {  // no centers, no edges: the gradient is zero
    hipLaunchKernelGGL(zero_floats_kernel, dim3(unsigned((cols + 255) / 256)), dim3(256), 0, s, cols, grad_path_w);
    return after_launch("allegro_tp_backward_train");
  }
  size_t need = 0;
  (void)allegro_tp_backward_workspace(plan, N, &need);
  if ((rc = check_tensor(workspace, "workspace"))) return rc;
  if (workspace_bytes < need)
    return fail(ALLEGRO_E_INVALID, "workspace of %zu bytes is smaller than the %zu required", workspace_bytes, need);
  if ((rc = check_tensor(grad_env, "grad_env")) || (rc = check_tensor(env, "env")) ||
      (rc = check_tensor(path_w, "path_w")))
    return rc;
  if (E > 0 && ((rc = check_tensor(x, "x")) || (rc = check_tensor(grad_out, "grad_out")) ||
                (rc = check_tensor(w, "w")) || (rc = check_tensor(Y, "Y")) || (rc = check_tensor(grad_x, "grad_x")) ||
                (rc = check_tensor(grad_w, "grad_w")) || (rc = check_tensor(grad_Y, "grad_Y"))))
    return rc;
  auto *mp = const_cast<allegro_tp_plan *>(plan);
  // validated: the status word stays locked from the CSR check to the report
  // of the handover waits
  const bool validate = (plan->flags & ALLEGRO_VALIDATE) != 0;
  std::unique_lock<std::mutex> vlock;
  if (validate) {
    vlock = std::unique_lock<std::mutex>(mp->validate_mu);
    if ((rc = validate_csr_locked(mp, N, E, row_ptr, s))) return rc;
  }
  const Kernels k = select(plan);
  if (!k.bwd_wg) return fail(ALLEGRO_E_UNSUPPORTED, "no kernel for this plan");
  float *part = static_cast<float *>(workspace);
  k.bwd_wg(dim3(unsigned(N)), s, row_ptr, x, env, path_w, grad_out, w, Y, grad_x, grad_env, grad_w, grad_Y, part,
           WaitCfg{plan->spin_limit, validate ? plan->status : nullptr});
  if ((rc = after_launch("allegro_tp_backward_train"))) return rc;
  const unsigned cb = unsigned((cols + 255) / 256);
  if (k.pw_rounds) {
    hipLaunchKernelGGL(pw_reduce_waves_kernel, dim3(cb), dim3(256), 0, s, int(k.pw_rounds(N)), plan->U,
                       int(plan->table.paths.size()), part, grad_path_w);
  } else {
    float *chunks = part + N * cols;
    hipLaunchKernelGGL(pw_reduce_rows_kernel, dim3(cb, kPwChunks), dim3(256), 0, s, N, cols, part, chunks);
    hipLaunchKernelGGL(pw_reduce_chunks_kernel, dim3(cb), dim3(256), 0, s, kPwChunks, cols, chunks, grad_path_w);
  }
  if ((rc = after_launch("allegro_tp_backward_train"))) return rc;
  return validate ? check_handover_locked(mp, s, "allegro_tp_backward_train") : ALLEGRO_OK;
}

int allegro_tp_backward_train_noalloc(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr,
                                      const float *x, const float *env, const float *path_w, const float *grad_out,
                                      const float *w, const float *Y, float *grad_x, float *grad_env, float *grad_w,
                                      float *grad_Y, float *grad_path_w, void *stream) {
  int rc = check_sizes(plan, N, E, row_ptr);
  if (rc) return rc;
  if ((rc = check_tensor(grad_path_w, "grad_path_w"))) return rc;
  const int cols = int(plan->table.paths.size()) * plan->U;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (N == 0) {  // no centers, no edges: the gradient is zero
    hipLaunchKernelGGL(zero_floats_kernel, dim3(unsigned((cols + 255) / 256)), dim3(256), 0, s, cols, grad_path_w);
    return after_launch("allegro_tp_backward_train_noalloc");
  }
  const Kernels k = select(plan);
  if (!k.bwd_wg) return fail(ALLEGRO_E_UNSUPPORTED, "no kernel for this plan");
  const NoAllocLayout lay = noalloc_layout(cols);
  const int64_t n_chunks = (N + lay.centers - 1) / lay.centers;
  if (!k.pw_rounds && (lay.centers < 1 || n_chunks > kNoAllocChunks))
    return fail(ALLEGRO_E_INVALID,
                "N=%lld centers exceed the allocation-free maximum of %lld for this plan (%d path-weight columns, "
                "%zu-byte static scratch)", (long long)N, (long long)lay.centers * kNoAllocChunks, cols,
                sizeof(float) * kNoAllocFloats);
  if ((rc = check_tensor(grad_env, "grad_env")) || (rc = check_tensor(env, "env")) ||
      (rc = check_tensor(path_w, "path_w")))
    return rc;
  if (E > 0 && ((rc = check_tensor(x, "x")) || (rc = check_tensor(grad_out, "grad_out")) ||
                (rc = check_tensor(w, "w")) || (rc = check_tensor(Y, "Y")) || (rc = check_tensor(grad_x, "grad_x")) ||
                (rc = check_tensor(grad_w, "grad_w")) || (rc = check_tensor(grad_Y, "grad_Y"))))
    return rc;
  float *scr = nullptr;
  if ((rc = noalloc_scratch(&scr))) return rc;
  auto *mp = const_cast<allegro_tp_plan *>(plan);
  const bool validate = (plan->flags & ALLEGRO_VALIDATE) != 0;
  std::unique_lock<std::mutex> vlock;
  if (validate) {
    vlock = std::unique_lock<std::mutex>(mp->validate_mu);
    if ((rc = validate_csr_locked(mp, N, E, row_ptr, s))) return rc;
  }
  const WaitCfg wcfg{plan->spin_limit, validate ? plan->status : nullptr};
  const unsigned cb = unsigned((cols + 255) / 256);
  if (k.pw_rounds) {
    // the matrix-core kernel's per-wave rows fit the scratch at any N
    static_assert(kNoAllocFloats >= int64_t(kMaxPwRounds) * 128 * 68, "per-wave rows fit the scratch");
    const int64_t rounds = k.pw_rounds(N);  // at most kMaxPwRounds
    k.bwd_wg(dim3(unsigned(N)), s, row_ptr, x, env, path_w, grad_out, w, Y, grad_x, grad_env, grad_w, grad_Y, scr,
             wcfg);
    hipLaunchKernelGGL(pw_reduce_waves_kernel, dim3(cb), dim3(256), 0, s, int(rounds), plan->U,
                       int(plan->table.paths.size()), scr, grad_path_w);
    if ((rc = after_launch("allegro_tp_backward_train_noalloc"))) return rc;
    return validate ? check_handover_locked(mp, s, "allegro_tp_backward_train_noalloc") : ALLEGRO_OK;
  }
  // scratch: per-center rows of one chunk, the 128 range sums of a chunk, then
  // one row per chunk; every region is fully written before it is read
  float *part = scr, *ranges = part + lay.centers * cols, *chunk_rows = ranges + int64_t(kPwChunks) * cols;
  const int64_t ud2 = int64_t(plan->U) * plan->table.d2;
  for (int64_t c = 0; c < n_chunks; ++c) {
    const int64_t n0 = c * lay.centers, n1 = std::min(N, n0 + lay.centers);
    // the chunk's centers as a CSR of their own: row_ptr values stay absolute
    // edge indices, center-indexed tensors are offset to the chunk's first center
    k.bwd_wg(dim3(unsigned(n1 - n0)), s, row_ptr + n0, x, env + n0 * ud2, path_w, grad_out, w, Y, grad_x,
             grad_env + n0 * ud2, grad_w, grad_Y, part, wcfg);
    hipLaunchKernelGGL(pw_reduce_rows_kernel, dim3(cb, kPwChunks), dim3(256), 0, s, n1 - n0, cols, part, ranges);
    hipLaunchKernelGGL(pw_reduce_chunks_kernel, dim3(cb), dim3(256), 0, s, kPwChunks, cols, ranges,
                       chunk_rows + c * cols);
    if ((rc = after_launch("allegro_tp_backward_train_noalloc"))) return rc;
  }
  hipLaunchKernelGGL(pw_reduce_chunks_kernel, dim3(cb), dim3(256), 0, s, int(n_chunks), cols, chunk_rows,
                     grad_path_w);
  if ((rc = after_launch("allegro_tp_backward_train_noalloc"))) return rc;
  return validate ? check_handover_locked(mp, s, "allegro_tp_backward_train_noalloc") : ALLEGRO_OK;
}

// One edge per thread in 256-thread blocks; the grid's x extent stays below 2^31.
constexpr int64_t kMaxShEdges = (int64_t(1) << 31) * 255;

int allegro_sh_forward(const allegro_tp_plan *plan, int64_t E, const double *vec, float *Y, void *stream) {
  if (!plan) return fail(ALLEGRO_E_INVALID, "plan is NULL");
  if (E < 0) return fail(ALLEGRO_E_INVALID, "negative size (E=%lld)", (long long)E);
  if (E == 0) return ALLEGRO_OK;
  if (E > kMaxShEdges) return fail(ALLEGRO_E_INVALID, "E=%lld exceeds the grid limit", (long long)E);
  int rc;
  if ((rc = check_tensor(vec, "vec")) || (rc = check_tensor(Y, "Y"))) return rc;
  const unsigned blocks = unsigned((E + 255) / 256);
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (plan->lmax) {
    case 1: hipLaunchKernelGGL(sh_forward_kernel<1>, dim3(blocks), dim3(256), 0, s, E, vec, Y); break;
    case 2: hipLaunchKernelGGL(sh_forward_kernel<2>, dim3(blocks), dim3(256), 0, s, E, vec, Y); break;
    case 3: hipLaunchKernelGGL(sh_forward_kernel<3>, dim3(blocks), dim3(256), 0, s, E, vec, Y); break;
    default: return fail(ALLEGRO_E_UNSUPPORTED, "lmax=%d", plan->lmax);
  }
  return after_launch("allegro_sh_forward");
}

int allegro_sh_backward(const allegro_tp_plan *plan, int64_t E, const double *vec, const float *grad_Y,
                        double *grad_vec, void *stream) {
  if (!plan) return fail(ALLEGRO_E_INVALID, "plan is NULL");
  if (E < 0) return fail(ALLEGRO_E_INVALID, "negative size (E=%lld)", (long long)E);
  if (E == 0) return ALLEGRO_OK;
  if (E > kMaxShEdges) return fail(ALLEGRO_E_INVALID, "E=%lld exceeds the grid limit", (long long)E);
  int rc;
  if ((rc = check_tensor(vec, "vec")) || (rc = check_tensor(grad_Y, "grad_Y")) ||
      (rc = check_tensor(grad_vec, "grad_vec")))
    return rc;
  const unsigned blocks = unsigned((E + 255) / 256);
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (plan->lmax) {
    case 1: hipLaunchKernelGGL(sh_backward_kernel<1>, dim3(blocks), dim3(256), 0, s, E, vec, grad_Y, grad_vec); break;
    case 2: hipLaunchKernelGGL(sh_backward_kernel<2>, dim3(blocks), dim3(256), 0, s, E, vec, grad_Y, grad_vec); break;
    case 3: hipLaunchKernelGGL(sh_backward_kernel<3>, dim3(blocks), dim3(256), 0, s, E, vec, grad_Y, grad_vec); break;
    default: return fail(ALLEGRO_E_UNSUPPORTED, "lmax=%d", plan->lmax);
  }
  return after_launch("allegro_sh_backward");
}

const char *allegro_last_error(void) { return allegro_internal::last_error(); }

}  // extern "C"
