// Page gather export and the calibration / placement probes.
//
// Gather: request r's logical keys or values, token t read from slot t % 16 of physical page
// page_table[r][t / 16] -- the same address arithmetic the attention kernels use, exported so
// a test can compare it bit for bit with an index gather on the host.
//
// Calibration probes (paper, Section 3 "Opportunity" and Section 4.2: achievable HBM bandwidth
// and compute throughput are profiled once per partition size):
//   read probe  -- every thread streams 16-byte loads over a buffer larger than the last-level
//                  cache and folds them into a checksum;
//   MFMA probe  -- independent chains of 16x16x32 bf16 MFMAs on register operands, two waves per
//                  SIMD (on this part that instruction reaches about 98% of the nominal rate,
//                  the 32x32x16 one about 80%, so this is the share's ceiling);
//   placement   -- each workgroup records the XCC_ID and HW_ID hardware registers, which tell
//                  on which XCD / shader engine / CU it ran, to check a stream's CU mask.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace duet {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename T>
__global__ __launch_bounds__(256) void gather_kernel(const T* cache, int which, int h_kv, int d,
                                                     const int32_t* page_table, int max_pages, long long num_phys,
                                                     int req, int kv_len, T* out, int32_t* err) {
  const long long n = (long long)kv_len * h_kv * d;
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < n; i += (long long)gridDim.x * 256) {
    const int e = (int)(i % d);
    const int jh = (int)((i / d) % h_kv);
    const int t = (int)(i / ((long long)d * h_kv));
    const int id = page_table[(size_t)req * max_pages + (t >> 4)];
    if (id < 0 || (long long)id >= num_phys) {
      atomicOr(err, 1);
      out[i] = T(0);
      continue;
    }
    const size_t slab = ((size_t)id * h_kv + jh) * 16 * d;
    out[i] = which == 0 ? cache[slab + (size_t)(t & 15) * d + e] : cache[slab + (size_t)e * 16 + (t & 15)];
  }
}

// Each wave streams its own contiguous chunk of the buffer (n16 / waves 16-byte words, rounded
// down to whole 1 KiB wave steps), four wave steps in flight per lane; a sequential run per wave
// is the access pattern DRAM serves best, so the probe measures the share's ceiling.
__global__ __launch_bounds__(256) void read_probe_kernel(const uint4* buf, size_t n16, unsigned* sink) {
  const size_t waves = (size_t)gridDim.x * 4;
  const size_t wave = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const size_t per_wave = (n16 / waves) & ~(size_t)255;  // whole groups of four 64-word steps
  const uint4* p = buf + wave * per_wave + lane;
  uint32_t acc = 0;
  for (size_t i = 0; i < per_wave; i += 256) {
    const uint4 a = p[i], b = p[i + 64], c = p[i + 128], d = p[i + 192];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  if (acc == 0x9e3779b9u) sink[0] = acc;  // keeps the loads alive; practically never stores
}

// One workgroup of 8 waves per CU (two per SIMD); each loop trip issues 32 MFMAs over the four
// chains, so loop overhead stays out of the measurement.
__global__ __launch_bounds__(512, 1) void mfma_probe_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = static_cast<__bf16>(0.001f * (lane + e));
    b[e] = static_cast<__bf16>(0.002f * (lane - e));
  }
  f32x4 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      c0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c3, 0, 0, 0);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int v = 0; v < 4; ++v) s += c0[v] + c1[v] + c2[v] + c3[v];
  if (s == 1234.5f) sink[0] = s;  // keeps the chains alive
}

// s_getreg immediates: size-1 in bits 15:11, offset in 10:6, register id in 5:0.
constexpr int kHwRegHwId = (31 << 11) | (0 << 6) | 4;   // HW_ID: wave, SIMD, CU, SH, SE ids
constexpr int kHwRegXccId = (15 << 11) | (0 << 6) | 20;  // XCC_ID: which XCD

__global__ __launch_bounds__(64) void placement_kernel(uint32_t* out) {
  if (threadIdx.x == 0) {
    out[2 * blockIdx.x + 0] = __builtin_amdgcn_s_getreg(kHwRegXccId);
    out[2 * blockIdx.x + 1] = __builtin_amdgcn_s_getreg(kHwRegHwId);
  }
  // Hold the CU for a bounded ~20 us so later workgroups spread to other CUs.
  const uint64_t t0 = wall_clock64();
  for (int i = 0; i < 100000; ++i) {
    if (wall_clock64() - t0 > 2000) break;  // 100 MHz wall clock: 2000 ticks = 20 us
    __builtin_amdgcn_s_sleep(2);
  }
}

}  // namespace

hipError_t launch_gather(const void* cache, int which, int elem_bytes, int h_kv, int d, const int32_t* page_table,
                         int max_pages, long long num_phys, int req, int kv_len, void* out, int32_t* err,
                         hipStream_t s) {
  const long long n = (long long)kv_len * h_kv * d;
  if (n == 0) return hipSuccess;
  const int blocks = (int)std::min<long long>((n + 255) / 256, 4096);
  if (elem_bytes == 2)
    hipLaunchKernelGGL(gather_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, (const uint16_t*)cache, which, h_kv, d,
                       page_table, max_pages, num_phys, req, kv_len, (uint16_t*)out, err);
  else
    hipLaunchKernelGGL(gather_kernel<uint32_t>, dim3(blocks), dim3(256), 0, s, (const uint32_t*)cache, which, h_kv, d,
                       page_table, max_pages, num_phys, req, kv_len, (uint32_t*)out, err);
  return hipGetLastError();
}

// Bytes the read probe reads with `blocks` workgroups over a buffer of `bytes`.
size_t read_probe_bytes(size_t bytes, int blocks) {
  const size_t waves = (size_t)blocks * 4;
  return ((bytes / 16 / waves) & ~(size_t)255) * waves * 16;
}

hipError_t launch_read_probe(const void* buf, size_t bytes, int blocks, unsigned* sink, hipStream_t s) {
  hipLaunchKernelGGL(read_probe_kernel, dim3(blocks), dim3(256), 0, s, (const uint4*)buf, bytes / 16, sink);
  return hipGetLastError();
}

hipError_t launch_mfma_probe(int blocks, int iters, float* sink, hipStream_t s) {
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(512), 0, s, iters, sink);
  return hipGetLastError();
}

hipError_t launch_placement_probe(int blocks, uint32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(placement_kernel, dim3(blocks), dim3(64), 0, s, out);
  return hipGetLastError();
}

}  // namespace duet
