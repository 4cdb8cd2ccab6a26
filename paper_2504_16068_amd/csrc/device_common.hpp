// Device helpers shared by the tensor-product and layer kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

namespace allegro_dev {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Streaming 16-byte accesses with the non-temporal hint: edge-major tensors
// are touched once per kernel, so they should not displace other lines in L2.
__device__ __forceinline__ float4 load_stream(const float4 *p) {
  const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void store_stream(float4 v, float4 *p) {
  const f32x4 w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, reinterpret_cast<f32x4 *>(p));
}

// Orders the LDS accesses of the H waves of a workgroup without waiting for
// their outstanding global memory operations (__syncthreads() also waits for
// every in-flight global store, which would serialise a tile pipeline).  A
// single wave executes its LDS operations in order, so for H == 1 only the
// compiler needs the fences.  No kernel here relies on a barrier for global
// memory visibility between threads.
template <int H>
__device__ __forceinline__ void lds_sync() {
  if constexpr (H == 1) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  }
}

// Calls f(std::integral_constant<int, C>{}) for C = BEGIN .. END - 1, so that
// the body can index register arrays with compile-time constants.
template <int BEGIN, int END, class F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (BEGIN < END) {
    f(std::integral_constant<int, BEGIN>{});
    static_for<BEGIN + 1, END>(f);
  }
}

}  // namespace allegro_dev
