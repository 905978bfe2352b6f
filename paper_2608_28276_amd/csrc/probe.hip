// On-device bandwidth probes for the benchmark (not part of the PASK C ABI):
// a streaming reader and a streaming copy, the ceilings a HBM-bound kernel of
// this library is compared with on the box that runs it.
//
//   pask_probe_read   reads n bytes once (16-byte non-temporal loads, eight
//                     in flight per lane, grid-stride) and folds them into one
//                     word per workgroup (so the loads cannot be dropped).
//   pask_probe_copy   copies n bytes (16-byte non-temporal loads and stores,
//                     eight in flight per lane, grid-stride).
// Eight loads in flight per lane read about 6% faster than four on MI355X
// (7.07 against 6.69 TB/s at 8 workgroups of 256 per compute unit), and
// non-temporal stores copy 10-20% faster than plain ones (5.37 against
// 4.47-4.55 TB/s), so these are the best of the variants measured.
// Both take 16-byte aligned buffers whose size is a multiple of 64 bytes;
// anything else is rejected before a launch.
#include <hip/hip_runtime.h>

#include <stddef.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 8;

__global__ __launch_bounds__(kThreads) void read_kernel(const u32x4_t* __restrict__ src, size_t n16,
                                                         uint32_t* __restrict__ out) {
  __shared__ uint32_t s_acc[kThreads / 64];
  const size_t stride = (size_t)gridDim.x * kThreads * kUnroll;
  uint32_t acc = 0u;
  for (size_t i = (size_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; i < n16; i += stride) {
    u32x4_t x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const size_t j = i + (size_t)u * kThreads;
      x[u] = j < n16 ? __builtin_nontemporal_load(src + j) : u32x4_t{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= x[u][0] ^ x[u][1] ^ x[u][2] ^ x[u][3];
  }
  for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) s_acc[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = s_acc[0] ^ s_acc[1] ^ s_acc[2] ^ s_acc[3];
}

__global__ __launch_bounds__(kThreads) void copy_kernel(const u32x4_t* __restrict__ src, u32x4_t* __restrict__ dst,
                                                         size_t n16) {
  const size_t stride = (size_t)gridDim.x * kThreads * kUnroll;
  for (size_t i = (size_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; i < n16; i += stride) {
    u32x4_t x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const size_t j = i + (size_t)u * kThreads;
      if (j < n16) x[u] = __builtin_nontemporal_load(src + j);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const size_t j = i + (size_t)u * kThreads;
      if (j < n16) __builtin_nontemporal_store(x[u], dst + j);
    }
  }
}

}  // namespace

extern "C" {

// Workgroups of the probes: `blocks` (at most 65535; 0 picks 8 per compute unit).
int pask_probe_blocks(int blocks) {
  if (blocks > 0) return blocks > 65535 ? 65535 : blocks;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return -1;
  return 8 * cus;
}

// out: device, one uint32 per workgroup (pask_probe_blocks(blocks) of them).
int pask_probe_read(const void* src, size_t n, uint32_t* out, int blocks, hipStream_t s) {
  if (!src || !out || (reinterpret_cast<uintptr_t>(src) & 15) || n % 64) return -1;
  const int g = pask_probe_blocks(blocks);
  if (g <= 0) return -1;
  read_kernel<<<dim3(g), dim3(kThreads), 0, s>>>(static_cast<const u32x4_t*>(src), n / 16, out);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

int pask_probe_copy(const void* src, void* dst, size_t n, int blocks, hipStream_t s) {
  if (!src || !dst || (reinterpret_cast<uintptr_t>(src) & 15) || (reinterpret_cast<uintptr_t>(dst) & 15) || n % 64)
    return -1;
  const int g = pask_probe_blocks(blocks);
  if (g <= 0) return -1;
  copy_kernel<<<dim3(g), dim3(kThreads), 0, s>>>(static_cast<const u32x4_t*>(src), static_cast<u32x4_t*>(dst),
                                                 n / 16);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // extern "C"
