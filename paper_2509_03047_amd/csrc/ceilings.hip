// Plain streaming kernels that measure what HBM delivers on this chip to
// the access patterns the restore kernels use: a copy, a read-only sweep and
// a write-only sweep, with 16-byte non-temporal accesses and 64-lane
// workgroups launched in address order.  The benchmark reports each
// operation of the restore path against the ceiling of its own traffic mix
// (pack and unpack: copy; replica compare and checksum: read-only).  Not
// part of the restore library: built as its own shared object and loaded by
// the benchmark only.
//
// Work per workgroup follows measurements on MI355X: a copy peaks with
// 1 KiB per workgroup (one vector per lane); a pure read or write stops near
// 4.9 TB/s at 1 KiB per workgroup (the dispatcher launches about 4.7
// workgroups per ns) and peaks with 4 KiB.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kLanes = 64;

__global__ __launch_bounds__(kLanes) void k_copy(const u32x4* __restrict__ src,
                                                 u32x4* __restrict__ dst, uint64_t n_vec) {
  const uint64_t v = uint64_t(blockIdx.x) * kLanes + threadIdx.x;
  if (v < n_vec) __builtin_nontemporal_store(__builtin_nontemporal_load(src + v), dst + v);
}

// Each workgroup reads 4 vectors per lane; the XOR of everything read is
// stored only when it equals `never` (a value the caller picks so that it
// does not occur), which keeps the loads without adding write traffic.
__global__ __launch_bounds__(kLanes) void k_read(const u32x4* __restrict__ src, uint64_t n_vec,
                                                 uint32_t never, uint32_t* __restrict__ sink) {
  const uint64_t base = uint64_t(blockIdx.x) * (4 * kLanes) + threadIdx.x;
  u32x4 x[4];
#pragma unroll
  for (int q = 0; q < 4; q++) {
    const uint64_t v = base + uint64_t(q) * kLanes;
    x[q] = v < n_vec ? __builtin_nontemporal_load(src + v) : u32x4{0, 0, 0, 0};
  }
  const u32x4 y = x[0] ^ x[1] ^ x[2] ^ x[3];
  const uint32_t r = y.x ^ y.y ^ y.z ^ y.w;
  if (r == never) sink[threadIdx.x] = r;
}

__global__ __launch_bounds__(kLanes) void k_write(u32x4* __restrict__ dst, uint64_t n_vec,
                                                  uint32_t value) {
  const uint64_t base = uint64_t(blockIdx.x) * (4 * kLanes) + threadIdx.x;
#pragma unroll
  for (int q = 0; q < 4; q++) {
    const uint64_t v = base + uint64_t(q) * kLanes;
    if (v < n_vec) __builtin_nontemporal_store(u32x4{value, value, value, value}, dst + v);
  }
}

bool ok_size(uint64_t bytes, uint64_t per_group) {
  return bytes % 16 == 0 && bytes / per_group < (uint64_t(1) << 31) / kLanes;
}

}  // namespace

// Each returns 0 or the HIP error of the launch; buffers are 16-byte aligned
// device memory of `bytes` bytes (a multiple of 16), `sink` 256 bytes.
extern "C" int frc_copy(void* dst, const void* src, uint64_t bytes, hipStream_t stream) {
  if (!ok_size(bytes, 1024)) return int(hipErrorInvalidValue);
  const uint64_t n_vec = bytes / 16;
  hipLaunchKernelGGL(k_copy, dim3(uint32_t((n_vec + kLanes - 1) / kLanes)), dim3(kLanes), 0, stream,
                     static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), n_vec);
  return int(hipGetLastError());
}

extern "C" int frc_read(const void* src, uint64_t bytes, uint32_t never, uint32_t* sink,
                        hipStream_t stream) {
  if (!ok_size(bytes, 4096)) return int(hipErrorInvalidValue);
  const uint64_t n_vec = bytes / 16;
  hipLaunchKernelGGL(k_read, dim3(uint32_t((n_vec + 4 * kLanes - 1) / (4 * kLanes))), dim3(kLanes), 0,
                     stream, static_cast<const u32x4*>(src), n_vec, never, sink);
  return int(hipGetLastError());
}

extern "C" int frc_write(void* dst, uint64_t bytes, uint32_t value, hipStream_t stream) {
  if (!ok_size(bytes, 4096)) return int(hipErrorInvalidValue);
  const uint64_t n_vec = bytes / 16;
  hipLaunchKernelGGL(k_write, dim3(uint32_t((n_vec + 4 * kLanes - 1) / (4 * kLanes))), dim3(kLanes), 0,
                     stream, static_cast<u32x4*>(dst), n_vec, value);
  return int(hipGetLastError());
}
