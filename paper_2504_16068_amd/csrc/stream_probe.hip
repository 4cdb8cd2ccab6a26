// Streaming probes for bench.py: the HBM rate of plain read-only,
// one-read-one-write and two-read-one-write streams on this GPU, measured in
// the same run as the kernels, so that each kernel's rate can be set against
// the rate of its own access pattern.  Non-temporal 16-byte accesses, as the
// tensor-product kernels use.  Not part of the library's ABI.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// PATTERN 0: read a (each thread writes one float of its sums to c)
//         1: c = a
//         2: c = a + b
// Each thread moves UNROLL float4 per tensor per iteration, the iterations
// striding over the whole grid.
template <int PATTERN, int UNROLL>
__global__ __launch_bounds__(256) void stream_kernel(const f32x4 *__restrict__ a, const f32x4 *__restrict__ b,
                                                     f32x4 *__restrict__ c, int64_t n) {
  const int64_t stride = int64_t(gridDim.x) * 256 * UNROLL;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t base = int64_t(blockIdx.x) * 256 * UNROLL + threadIdx.x; base < n; base += stride) {
    f32x4 va[UNROLL], vb[UNROLL];
#pragma unroll
    for (int k = 0; k < UNROLL; ++k) {
      const int64_t i = base + int64_t(k) * 256;
      if (i < n) {
        va[k] = __builtin_nontemporal_load(a + i);
        if constexpr (PATTERN == 2) vb[k] = __builtin_nontemporal_load(b + i);
      }
    }
#pragma unroll
    for (int k = 0; k < UNROLL; ++k) {
      const int64_t i = base + int64_t(k) * 256;
      if (i < n) {
        if constexpr (PATTERN == 0) acc += va[k];
        if constexpr (PATTERN == 1) __builtin_nontemporal_store(va[k], c + i);
        if constexpr (PATTERN == 2) __builtin_nontemporal_store(va[k] + vb[k], c + i);
      }
    }
  }
  if constexpr (PATTERN == 0) reinterpret_cast<float *>(c)[int64_t(blockIdx.x) * 256 + threadIdx.x] =
      acc.x + acc.y + acc.z + acc.w;
}

template <int PATTERN>
void launch(int unroll, unsigned blocks, hipStream_t s, const f32x4 *a, const f32x4 *b, f32x4 *c, int64_t n) {
  if (unroll == 1) hipLaunchKernelGGL((stream_kernel<PATTERN, 1>), dim3(blocks), dim3(256), 0, s, a, b, c, n);
  else if (unroll == 2) hipLaunchKernelGGL((stream_kernel<PATTERN, 2>), dim3(blocks), dim3(256), 0, s, a, b, c, n);
  else hipLaunchKernelGGL((stream_kernel<PATTERN, 4>), dim3(blocks), dim3(256), 0, s, a, b, c, n);
}

// Access pattern of the lmax-3 matrix-core backward's tile stream, without its
// arithmetic: c = a + b over tensors [E][U][32] (fp32), a persistent grid of
// workgroups of 8 waves, each wave walking its own sequence of (center,
// channel group) pairs round robin, 16 edges per tile, DEPTH tiles loaded
// before they are stored, ROWF4 float4 of an edge's row per wave (8: one
// channel of 32 floats, 128 bytes; 16: two; 32: four).  Rows past a center's
// edges lie past the buffer descriptor's range: loads read zeros, stores drop.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), short(0), int(bytes), 0x00020000);
}

template <int ROWF4, int DEPTH>
__global__ __launch_bounds__(512) void pattern_kernel(int64_t N, int U, const int64_t *__restrict__ row_ptr,
                                                      const float *__restrict__ a, const float *__restrict__ b,
                                                      float *__restrict__ c) {
  constexpr int LR = 64 / ROWF4;  // rows per 16-byte load instruction
  constexpr int LJ = 16 / LR;     // load instructions per tensor and tile
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / 64), lane = int(threadIdx.x) % 64;
  const int groups = U * 8 / ROWF4;  // channel groups per center (8 float4 per channel)
  const int64_t total = int64_t(gridDim.x) * 8, pairs = N * groups;
  const uint32_t row_bytes = uint32_t(U) * 128u;
  const uint32_t voff = uint32_t(lane / ROWF4) * row_bytes + uint32_t(lane % ROWF4) * 16u;
  for (int64_t fq = int64_t(blockIdx.x) * 8 + wave; fq < pairs; fq += total) {
    const int64_t n = fq / groups;
    const int gi = int(fq % groups);
    const int64_t e0 = row_ptr[n], e1 = row_ptr[n + 1];
    for (int64_t e = e0; e < e1; e += 16 * DEPTH) {
      f32x4 va[DEPTH][LJ], vb[DEPTH][LJ];
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        const int64_t te = e + 16 * d;
        const uint32_t bytes = te < e1 ? uint32_t(e1 - te < 16 ? e1 - te : 16) * row_bytes : 0u;
        const int64_t base = te * U * 32 + int64_t(gi) * ROWF4 * 4;
        const auto ra = row_rsrc(a + base, bytes), rb = row_rsrc(b + base, bytes);
#pragma unroll
        for (int j = 0; j < LJ; ++j) {
          const int o = int(voff + uint32_t(LR * j) * row_bytes);
          va[d][j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, o, 0, 2));
          vb[d][j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rb, o, 0, 2));
        }
      }
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        const int64_t te = e + 16 * d;
        const uint32_t bytes = te < e1 ? uint32_t(e1 - te < 16 ? e1 - te : 16) * row_bytes : 0u;
        const auto rc = row_rsrc(c + te * U * 32 + int64_t(gi) * ROWF4 * 4, bytes);
#pragma unroll
        for (int j = 0; j < LJ; ++j)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, va[d][j] + vb[d][j]), rc,
                                                 int(voff + uint32_t(LR * j) * row_bytes), 0, 2);
      }
    }
  }
}

// A plain copy out = x of edge rows of RF4 float4 with the direct kernels'
// traversal: one workgroup of NW waves per center, each wave copying whole
// edge rows of its center round robin (non-temporal 16-byte accesses).
template <int NW, int RF4>
__global__ __launch_bounds__(64 * NW) void center_copy_kernel(const int64_t *__restrict__ row_ptr,
                                                              const f32x4 *__restrict__ x, f32x4 *__restrict__ out) {
  constexpr int PER = (RF4 + 63) / 64;
  const int wave = int(threadIdx.x) / 64, lane = int(threadIdx.x) % 64;
  const int64_t n = blockIdx.x, e0 = row_ptr[n], e1 = row_ptr[n + 1];
  for (int64_t e = e0 + wave; e < e1; e += NW) {
    f32x4 v[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = lane + 64 * i;
      if (f < RF4) v[i] = __builtin_nontemporal_load(x + e * RF4 + f);
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = lane + 64 * i;
      if (f < RF4) __builtin_nontemporal_store(v[i], out + e * RF4 + f);
    }
  }
}

}  // namespace

// The per-center copy probe: rows of U * 18 floats (U = 64: 288 float4, the
// headline's x rows), one workgroup of 16 waves per center for N centers.
// Returns 0, -1 for bad arguments, -3 on a launch error.
extern "C" int center_copy_probe(int64_t N, const int64_t *row_ptr, const void *x, void *out, void *stream) {
  if (N <= 0 || !row_ptr || !x || !out) return -1;
  hipLaunchKernelGGL((center_copy_kernel<16, 288>), dim3(unsigned(N)), dim3(1024), 0, static_cast<hipStream_t>(stream),
                     row_ptr, static_cast<const f32x4 *>(x), static_cast<f32x4 *>(out));
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// The access-pattern probe: variant 0 = 128-byte rows, 4 tiles in flight;
// 1 = 128-byte rows, 6 tiles; 2 = 256-byte rows, 2 tiles; 3 = 256-byte rows,
// 4 tiles; 4 = 512-byte rows, 2 tiles.  a, b, c hold row_ptr[N] rows of
// U * 32 floats; U is 64 or 128.  Returns 0, -1 for bad arguments, -3 on a
// launch error.
extern "C" int pattern_probe(int variant, int64_t N, int U, const int64_t *row_ptr, const void *a, const void *b,
                             void *c, unsigned blocks, void *stream) {
  if (N <= 0 || (U != 64 && U != 128) || !row_ptr || !a || !b || !c || blocks == 0) return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float *pa = static_cast<const float *>(a), *pb = static_cast<const float *>(b);
  float *pc = static_cast<float *>(c);
  switch (variant) {
    case 0: hipLaunchKernelGGL((pattern_kernel<8, 4>), dim3(blocks), dim3(512), 0, s, N, U, row_ptr, pa, pb, pc); break;
    case 1: hipLaunchKernelGGL((pattern_kernel<8, 6>), dim3(blocks), dim3(512), 0, s, N, U, row_ptr, pa, pb, pc); break;
    case 2: hipLaunchKernelGGL((pattern_kernel<16, 2>), dim3(blocks), dim3(512), 0, s, N, U, row_ptr, pa, pb, pc); break;
    case 3: hipLaunchKernelGGL((pattern_kernel<16, 4>), dim3(blocks), dim3(512), 0, s, N, U, row_ptr, pa, pb, pc); break;
    case 4: hipLaunchKernelGGL((pattern_kernel<32, 2>), dim3(blocks), dim3(512), 0, s, N, U, row_ptr, pa, pb, pc); break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// n_f4 float4 per stream; blocks of 256 threads (for pattern 0, c must hold
// blocks * 256 floats).  Returns 0, or -1 for bad arguments, -3 on a launch
// error.
extern "C" int stream_probe(int pattern, int unroll, unsigned blocks, const void *a, const void *b, void *c,
                            int64_t n_f4, void *stream) {
  if (pattern < 0 || pattern > 2 || (unroll != 1 && unroll != 2 && unroll != 4) || blocks == 0 || n_f4 <= 0 ||
      !a || !c || (pattern == 2 && !b))
    return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const f32x4 *pa = static_cast<const f32x4 *>(a), *pb = static_cast<const f32x4 *>(b);
  f32x4 *pc = static_cast<f32x4 *>(c);
  switch (pattern) {
    case 0: launch<0>(unroll, blocks, s, pa, pb, pc, n_f4); break;
    case 1: launch<1>(unroll, blocks, s, pa, pb, pc, n_f4); break;
    default: launch<2>(unroll, blocks, s, pa, pb, pc, n_f4); break;
  }
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
