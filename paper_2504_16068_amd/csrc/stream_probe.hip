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

}  // namespace

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
