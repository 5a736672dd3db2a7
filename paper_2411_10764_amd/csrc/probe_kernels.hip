// Microbenchmarks behind the walks' roofline figures: LDS read throughput
// (consecutive and random 4-, 8- and 16-byte reads per lane) and 32-bit
// integer add throughput.  They measure the units the tree walks use; they
// are not part of scoring.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ml2_internal.h"

namespace {

constexpr int kProbeThreads = 256;
constexpr uint32_t kProbeLds = 65536;         // bytes of LDS each workgroup reads
constexpr uint32_t kProbeMask = kProbeLds - 16u;  // keeps every 16-byte read inside

// 32-bit integer hash: the xorshift-multiply "lowbias32" constants found by
// C. Wellons' hash-prospector search (2018).
__device__ __forceinline__ uint32_t mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// Eight reads per lane and iteration.  MODE 0..2: lane l of a wave reads
// bytes l * width onward of a 1 KiB window that moves by 64 bytes per
// iteration (consecutive addresses); MODE 3..5: hashed addresses, aligned to
// the read width.  Every address is masked into the 64 KiB buffer.
template <int MODE>
__global__ void __launch_bounds__(kProbeThreads) lds_probe_kernel(uint32_t *out, int iters) {
  __shared__ __attribute__((aligned(16))) char buf[kProbeLds];
  constexpr uint32_t width = 4u << (MODE % 3);
  const uint32_t tid = threadIdx.x, lane = tid & 63u;
  for (uint32_t i = tid; i < kProbeLds / 4u; i += kProbeThreads)
    reinterpret_cast<uint32_t *>(buf)[i] = mix(i);
  __syncthreads();
  uint32_t acc = 0;
  const uint32_t base = (tid >> 6) * 4096u;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      uint32_t a = MODE < 3 ? base + lane * width + (uint32_t)k * 1024u + (uint32_t)it * 64u
                            : mix(lane * 131u + (uint32_t)k * 7u + (uint32_t)it * 977u);
      a &= kProbeMask & ~(width - 1u);
      if constexpr (width == 4) {
        acc ^= *reinterpret_cast<const uint32_t *>(buf + a);
      } else if constexpr (width == 8) {
        const uint2 v = *reinterpret_cast<const uint2 *>(buf + a);
        acc ^= v.x ^ v.y;
      } else {
        const uint4 v = *reinterpret_cast<const uint4 *>(buf + a);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
      }
    }
  }
  out[blockIdx.x * kProbeThreads + tid] = acc;
}

// Eight independent chains of 32-bit adds per lane, 16 adds each per
// iteration (inline so that the compiler keeps every add).
__global__ void __launch_bounds__(kProbeThreads) valu_probe_kernel(uint32_t *out, int iters) {
  uint32_t a[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) a[c] = threadIdx.x + 7u * c;
  const uint32_t d = blockIdx.x | 1u;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
#pragma unroll
      for (int c = 0; c < 8; ++c) asm volatile("v_add_u32 %0, %0, %1" : "+v"(a[c]) : "v"(d));
    }
  }
  uint32_t x = 0;
#pragma unroll
  for (int c = 0; c < 8; ++c) x ^= a[c];
  out[blockIdx.x * kProbeThreads + threadIdx.x] = x;
}

}  // namespace

namespace ml2 {

hipError_t launch_lds_probe(int mode, int iters, int blocks, uint32_t *out, double *work,
                            hipStream_t s) {
  const dim3 grid(blocks), block(kProbeThreads);
  switch (mode) {
    case 0: hipLaunchKernelGGL(lds_probe_kernel<0>, grid, block, 0, s, out, iters); break;
    case 1: hipLaunchKernelGGL(lds_probe_kernel<1>, grid, block, 0, s, out, iters); break;
    case 2: hipLaunchKernelGGL(lds_probe_kernel<2>, grid, block, 0, s, out, iters); break;
    case 3: hipLaunchKernelGGL(lds_probe_kernel<3>, grid, block, 0, s, out, iters); break;
    case 4: hipLaunchKernelGGL(lds_probe_kernel<4>, grid, block, 0, s, out, iters); break;
    case 5: hipLaunchKernelGGL(lds_probe_kernel<5>, grid, block, 0, s, out, iters); break;
    default: return hipErrorInvalidValue;
  }
  const double width = 4u << (mode % 3);
  *work = (double)blocks * kProbeThreads * iters * 8.0 * width;  // bytes read
  return hipGetLastError();
}

hipError_t launch_valu_probe(int iters, int blocks, uint32_t *out, double *work, hipStream_t s) {
  hipLaunchKernelGGL(valu_probe_kernel, dim3(blocks), dim3(kProbeThreads), 0, s, out, iters);
  *work = (double)blocks * kProbeThreads * iters * 16.0 * 8.0;  // lane additions
  return hipGetLastError();
}

}  // namespace ml2
