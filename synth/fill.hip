// Device fill of a flat buffer with the seeded values of gen.h.
// It knows nothing of layouts: element idx of the buffer gets value(seed, stream, idx).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gen.h"

namespace {

template <typename T>
__device__ inline T value_at(uint64_t seed, uint64_t stream, uint64_t idx);

template <>
__device__ inline double value_at<double>(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_f64(seed, stream, idx);
}
template <>
__device__ inline float value_at<float>(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_f32(seed, stream, idx);
}
template <>
__device__ inline double2 value_at<double2>(uint64_t seed, uint64_t stream, uint64_t idx) {
  return make_double2(synth_c128_re(seed, stream, idx), synth_c128_im(seed, stream, idx));
}
template <>
__device__ inline float2 value_at<float2>(uint64_t seed, uint64_t stream, uint64_t idx) {
  return make_float2(synth_c64_re(seed, stream, idx), synth_c64_im(seed, stream, idx));
}

template <typename T>
__global__ void __launch_bounds__(256) fill_kernel(T* __restrict__ dst, uint64_t n, uint64_t seed,
                                                   uint64_t stream) {
  const uint64_t step = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += step)
    dst[i] = value_at<T>(seed, stream, i);
}

template <typename T>
int launch(void* dst, uint64_t n, uint64_t seed, uint64_t stream, hipStream_t s) {
  if (n == 0) return 0;
  uint64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s, (T*)dst, n, seed, stream);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // namespace

// dtype: 0 = f64, 1 = complex128, 2 = f32, 3 = complex64.  Returns 0 on success,
// 1 for an unknown dtype or a null pointer with n > 0, 2 for a HIP launch error.
extern "C" int synth_fill(int dtype, void* dst, uint64_t n, uint64_t seed, uint64_t stream,
                          hipStream_t s) {
  if (n > 0 && dst == nullptr) return 1;
  switch (dtype) {
    case 0: return launch<double>(dst, n, seed, stream, s);
    case 1: return launch<double2>(dst, n, seed, stream, s);
    case 2: return launch<float>(dst, n, seed, stream, s);
    case 3: return launch<float2>(dst, n, seed, stream, s);
    default: return 1;
  }
}

// Host fill with the same values (for host-side buffers of the CPU baseline).
extern "C" int synth_fill_host(int dtype, void* dst, uint64_t n, uint64_t seed, uint64_t stream) {
  if (n > 0 && dst == nullptr) return 1;
  switch (dtype) {
    case 0: {
      double* p = (double*)dst;
      for (uint64_t i = 0; i < n; ++i) p[i] = synth_f64(seed, stream, i);
      return 0;
    }
    case 1: {
      double* p = (double*)dst;
      for (uint64_t i = 0; i < n; ++i) {
        p[2 * i] = synth_c128_re(seed, stream, i);
        p[2 * i + 1] = synth_c128_im(seed, stream, i);
      }
      return 0;
    }
    case 2: {
      float* p = (float*)dst;
      for (uint64_t i = 0; i < n; ++i) p[i] = synth_f32(seed, stream, i);
      return 0;
    }
    case 3: {
      float* p = (float*)dst;
      for (uint64_t i = 0; i < n; ++i) {
        p[2 * i] = synth_c64_re(seed, stream, i);
        p[2 * i + 1] = synth_c64_im(seed, stream, i);
      }
      return 0;
    }
    default: return 1;
  }
}

// Host fill of elements [first, first + n) of a buffer: dst[i] gets the value of
// element first + i (so that several threads can fill one buffer in parts).
extern "C" int synth_fill_host_range(int dtype, void* dst, uint64_t first, uint64_t n, uint64_t seed,
                                     uint64_t stream) {
  if (n > 0 && dst == nullptr) return 1;
  switch (dtype) {
    case 0: {
      double* p = (double*)dst;
      for (uint64_t i = 0; i < n; ++i) p[i] = synth_f64(seed, stream, first + i);
      return 0;
    }
    case 1: {
      double* p = (double*)dst;
      for (uint64_t i = 0; i < n; ++i) {
        p[2 * i] = synth_c128_re(seed, stream, first + i);
        p[2 * i + 1] = synth_c128_im(seed, stream, first + i);
      }
      return 0;
    }
    case 2: {
      float* p = (float*)dst;
      for (uint64_t i = 0; i < n; ++i) p[i] = synth_f32(seed, stream, first + i);
      return 0;
    }
    case 3: {
      float* p = (float*)dst;
      for (uint64_t i = 0; i < n; ++i) {
        p[2 * i] = synth_c64_re(seed, stream, first + i);
        p[2 * i + 1] = synth_c64_im(seed, stream, first + i);
      }
      return 0;
    }
    default: return 1;
  }
}
