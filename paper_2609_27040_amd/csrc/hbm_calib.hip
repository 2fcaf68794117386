// Calibration kernels: what this GPU's HBM gives a plain streaming read and a
// plain streaming copy, measured beside the library's own kernels. They are
// built into a library of their own (libema_calib.so) that only the
// benchmark loads; nothing in libema_slice.so calls them.
//
// Both stream 16-byte non-temporal accesses in 4 KiB chunks, one per
// wavefront, four wavefronts a workgroup, every wavefront keeping its whole
// chunk in flight before it uses any of it (the read folds its chunk into one
// word so the loads are live; the copy stores it). Contiguous chunks,
// consecutive wavefronts on consecutive chunks: the best case for HBM, which
// is the point. (Of the chunk sizes and workgroup shapes tried, 2-16 KiB per
// wavefront with one or four wavefronts a workgroup, this one is at or near
// the best for both.)
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kLoads = 4;                 // 16 B each per lane: 4 KiB per wavefront
constexpr size_t kChunk = size_t(kLoads) * 64 * 16;
constexpr size_t kPerGroup = kChunk * kWaves;

__global__ __launch_bounds__(256) void calib_read_kernel(const char* __restrict__ src,
                                                         uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const size_t chunk = size_t(blockIdx.x) * kWaves + (threadIdx.x >> 6);
  const char* p = src + chunk * kChunk + lane * 16;
  u32x4 v[kLoads];
#pragma unroll
  for (int i = 0; i < kLoads; ++i)
    v[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p + size_t(i) * 1024));
  uint32_t x = 0;
#pragma unroll
  for (int i = 0; i < kLoads; ++i) x ^= v[i].x ^ v[i].y ^ v[i].z ^ v[i].w;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
  if (lane == 0) sink[chunk] = x;
}

__global__ __launch_bounds__(256) void calib_copy_kernel(const char* __restrict__ src,
                                                         char* __restrict__ dst) {
  const int lane = threadIdx.x & 63;
  const size_t off = (size_t(blockIdx.x) * kWaves + (threadIdx.x >> 6)) * kChunk + lane * 16;
  u32x4 v[kLoads];
#pragma unroll
  for (int i = 0; i < kLoads; ++i)
    v[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + off + size_t(i) * 1024));
#pragma unroll
  for (int i = 0; i < kLoads; ++i)
    __builtin_nontemporal_store(v[i], reinterpret_cast<u32x4*>(dst + off + size_t(i) * 1024));
}

}  // namespace

extern "C" {

// Reads src[bytes] (device) once; sink (device uint32 [bytes / 4096]) gets
// the XOR of each 4 KiB chunk's words. bytes must be a positive multiple of
// 16 KiB. Returns 0, -1 for bad arguments (nothing launched), or the HIP
// error of the launch.
int ema_calib_read(const void* src, size_t bytes, uint32_t* sink, void* stream) {
  if (!src || !sink || bytes == 0 || bytes % kPerGroup || bytes / kPerGroup > 0x7fffffffu)
    return -1;
  hipLaunchKernelGGL(calib_read_kernel, dim3(unsigned(bytes / kPerGroup)), dim3(kWaves * 64), 0,
                     static_cast<hipStream_t>(stream), static_cast<const char*>(src), sink);
  return int(hipGetLastError());
}

// dst[bytes] <- src[bytes] (device, not overlapping). bytes must be a positive
// multiple of 16 KiB. Returns 0, -1 for bad arguments (nothing launched), or
// the HIP error of the launch.
int ema_calib_copy(const void* src, void* dst, size_t bytes, void* stream) {
  if (!src || !dst || bytes == 0 || bytes % kPerGroup || bytes / kPerGroup > 0x7fffffffu)
    return -1;
  hipLaunchKernelGGL(calib_copy_kernel, dim3(unsigned(bytes / kPerGroup)), dim3(kWaves * 64), 0,
                     static_cast<hipStream_t>(stream), static_cast<const char*>(src),
                     static_cast<char*>(dst));
  return int(hipGetLastError());
}

}  // extern "C"
