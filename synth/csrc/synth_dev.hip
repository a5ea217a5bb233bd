// Seeded synthetic workload generator, device part (C ABI).
//
// Test and benchmark infrastructure only: fills device tables with the same
// counter-based normal values that synth_host.cpp draws on the CPU (both
// include synth_rng.h), so tables of many GiB never have to be drawn on the
// host and copied.  None of the phrase-memory method lives here.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <stdio.h>

#include "synth_rng.h"

// A launch is checked with hipGetLastError, which also reports a failed HIP
// call made earlier on this thread by other code: that status is cleared
// before the launch (and named on stderr, with the launch's own error).
static void clear_stale_status(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    fprintf(stderr, "synth: %s: earlier HIP status %s cleared before the launch\n", what,
            hipGetErrorName(e));
}

static int launched(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return 0;
  fprintf(stderr, "synth: %s launch failed: %s\n", what, hipGetErrorName(e));
  return -2;
}

// One thread per element of rows [row0, row0 + nrows); out points at row0.
template <int DT>
__global__ void k_normal_fill(void* __restrict__ out, int64_t row0, int64_t nrows, int64_t cols,
                              uint64_t key, float scale) {
  const int64_t n = nrows * cols;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t e = (uint64_t)row0 * (uint64_t)cols + (uint64_t)i;
    const float x = (float)synth_irwin_hall_n(key, e) * scale;
    if (DT == 0) ((float*)out)[i] = x;
    else ((uint16_t*)out)[i] = synth_f32_to_bf16(x);
  }
}

extern "C" int synth_normal_fill_dev(void* out, int64_t row0, int64_t nrows, int64_t cols,
                                     uint64_t key, float scale, int dtype, hipStream_t stream) {
  if (!out || nrows < 0 || cols <= 0 || (dtype != 0 && dtype != 1)) return -1;
  if (nrows == 0) return 0;
  const int64_t n = nrows * cols;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1 << 20) blocks = 1 << 20;
  clear_stale_status("normal fill");
  if (dtype == 0)
    hipLaunchKernelGGL(k_normal_fill<0>, dim3((unsigned)blocks), dim3(256), 0, stream, out, row0,
                       nrows, cols, key, scale);
  else
    hipLaunchKernelGGL(k_normal_fill<1>, dim3((unsigned)blocks), dim3(256), 0, stream, out, row0,
                       nrows, cols, key, scale);
  return launched("normal fill");
}

// Plain device copy (16 bytes per lane, non-temporal), used only as the
// bandwidth reference next to the lookup kernel: its HBM bytes are known
// exactly, which calibrates the profiler's fetch/write counters.
typedef uint32_t synth_u32x4 __attribute__((ext_vector_type(4)));

__global__ void k_copy16(const synth_u32x4* __restrict__ src, synth_u32x4* __restrict__ dst,
                         int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

extern "C" int synth_copy_dev(void* dst, const void* src, int64_t nbytes, int blocks,
                              hipStream_t stream) {
  if (!dst || !src || nbytes <= 0 || (nbytes & 15) || blocks <= 0) return -1;
  clear_stale_status("copy");
  hipLaunchKernelGGL(k_copy16, dim3((unsigned)blocks), dim3(256), 0, stream, (const synth_u32x4*)src,
                     (synth_u32x4*)dst, nbytes / 16);
  return launched("copy");
}

// Device address of pinned host memory (hipHostMalloc), so that the device
// filler can draw value tables straight into host memory.
extern "C" int synth_host_device_ptr(void* host, void** dev) {
  return hipHostGetDevicePointer(dev, host, 0) == hipSuccess ? 0 : -1;
}

// Busy-waits `us` microseconds on the device (bounded by the 100 MHz
// real-time counter and an iteration cap), standing in for the transformer
// layers that run between an early-exit prefetch and the next lookup.
__global__ void k_spin(uint64_t ticks) {
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  for (uint32_t it = 0; it < (1u << 26); ++it) {
    if (__builtin_amdgcn_s_memrealtime() - t0 >= ticks) break;
    __builtin_amdgcn_s_sleep(1);
  }
}

extern "C" int synth_spin_dev(double us, hipStream_t stream) {
  if (!(us >= 0.0) || us > 1e5) return -1;
  clear_stale_status("spin");
  hipLaunchKernelGGL(k_spin, dim3(1), dim3(64), 0, stream, (uint64_t)(us * 100.0));
  return launched("spin");
}
