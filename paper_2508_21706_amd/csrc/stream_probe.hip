// Streaming-read probe for MI355X (gfx950): the measured HBM read ceiling that
// the verification-attention kernel's bandwidth is compared with.
//
// Not part of the attention library: it is built into its own shared library
// (libspecmoe_probe.so) and used only by the benchmark.  It reads two
// contiguous byte ranges -- the benchmark hands it the same number of K and V
// bytes that one attention call streams -- with one persistent workgroup per
// CU, each taking an equal contiguous share of the concatenated ranges, with
// 16-byte non-temporal loads (the cache policy of the attention kernel's K/V
// tile loads) and about 128 KB in flight per CU.  Two ways of landing the
// bytes are measured:
//   mode 0: direct-to-LDS loads (global_load_lds), as the attention kernel's
//           producer waves issue them: 12 waves, each keeping 16 loads of
//           1 KB in flight, re-issued after its own s_waitcnt;
//   mode 1: plain loads into registers: each of 1024 threads keeps eight
//           16-byte loads in flight and folds them into an XOR, so that no
//           load can be dropped.
// Every workgroup writes one 32-bit word of its XOR (mode 1) or 0 (mode 0)
// to sink[blockIdx.x]; sink must hold `grid` words.
//
// C ABI (host):
//   int specmoe_probe_stream(const void* a, size_t a_bytes, const void* b,
//                            size_t b_bytes, int mode, int grid,
//                            uint32_t* sink, void* stream);
// a, b: device, 16-byte aligned, byte counts multiples of 16 (b may be NULL
// with b_bytes 0); grid in [1, 4096]; returns 0, or -1 for bad arguments and
// -2 when HIP reports a launch error.
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

constexpr int kStreaming = 2;   // non-temporal cache policy
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

struct ProbeArgs {
  const char* a;
  const char* b;
  uint64_t na, nb;   // bytes, multiples of 16
  uint32_t* sink;
};

// Byte range [lo, hi) of the concatenation a ++ b for workgroup w of P,
// rounded to 1 KB so that every load covers whole 64-byte lines.
__device__ __forceinline__ void share(const ProbeArgs& p, int w, int P, uint64_t& lo, uint64_t& hi) {
  const uint64_t n = p.na + p.nb;
  const uint64_t kb = (n + 1023) / 1024;
  lo = kb * (uint64_t)w / (uint64_t)P * 1024;
  hi = kb * (uint64_t)(w + 1) / (uint64_t)P * 1024;
  if (hi > n) hi = n;
  if (lo > n) lo = n;
}

// address of byte x of a ++ b (x < na + nb)
__device__ __forceinline__ const char* at(const ProbeArgs& p, uint64_t x) {
  return x < p.na ? p.a + x : p.b + (x - p.na);
}

constexpr int kLdsWaves = 12;
constexpr int kLdsLoads = 16;   // 1 KB loads in flight per wave

__global__ __launch_bounds__(64 * kLdsWaves, 1) void probe_lds_kernel(ProbeArgs p) {
  __shared__ __attribute__((aligned(16))) char buf[kLdsWaves * kLdsLoads * 1024 / 2];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  uint64_t lo, hi;
  share(p, blockIdx.x, gridDim.x, lo, hi);
  // loads alternate between the two halves of the wave's LDS region: the
  // bytes are not used, only landed
  char* mine = buf + wave * (kLdsLoads / 2) * 1024;
  const uint64_t step = (uint64_t)kLdsWaves * kLdsLoads * 1024;
  for (uint64_t base = lo + (uint64_t)wave * kLdsLoads * 1024; base < hi; base += step) {
#pragma unroll
    for (int k = 0; k < kLdsLoads; ++k) {
      const uint64_t x = base + (uint64_t)k * 1024 + 16u * lane;
      if (x < hi)
        __builtin_amdgcn_global_load_lds(at(p, x), (__attribute__((address_space(3))) void*)(mine + (k & 7) * 1024),
                                         16, 0, kStreaming);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  if (threadIdx.x == 0) p.sink[blockIdx.x] = 0u;
}

constexpr int kRegThreads = 1024;
constexpr int kRegLoads = 8;

__global__ __launch_bounds__(kRegThreads, 1) void probe_reg_kernel(ProbeArgs p) {
  uint64_t lo, hi;
  share(p, blockIdx.x, gridDim.x, lo, hi);
  u32x4 acc = {0u, 0u, 0u, 0u};
  const uint64_t step = (uint64_t)kRegThreads * kRegLoads * 16;
  for (uint64_t base = lo + 16u * threadIdx.x; base < hi; base += step) {
    u32x4 x[kRegLoads];
#pragma unroll
    for (int k = 0; k < kRegLoads; ++k) {
      const uint64_t y = base + (uint64_t)k * kRegThreads * 16;
      x[k] = y < hi ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(at(p, y))) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int k = 0; k < kRegLoads; ++k) acc ^= x[k];
  }
  __shared__ uint32_t red[kRegThreads / 64];
  uint32_t v = acc.x ^ acc.y ^ acc.z ^ acc.w;
  for (int off = 32; off > 0; off >>= 1) v ^= __shfl_xor(v, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0;
    for (int i = 0; i < kRegThreads / 64; ++i) r ^= red[i];
    p.sink[blockIdx.x] = r;
  }
}

}  // namespace

extern "C" int specmoe_probe_stream(const void* a, size_t a_bytes, const void* b, size_t b_bytes, int mode, int grid,
                                    uint32_t* sink, void* stream) {
  if (!a || !sink || (b_bytes && !b)) return -1;
  if ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) | a_bytes | b_bytes) & 15u) return -1;
  if (grid < 1 || grid > 4096 || (mode != 0 && mode != 1)) return -1;
  ProbeArgs p{static_cast<const char*>(a), static_cast<const char*>(b), a_bytes, b_bytes, sink};
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (mode == 0) hipLaunchKernelGGL(probe_lds_kernel, dim3(grid), dim3(64 * kLdsWaves), 0, s, p);
  else hipLaunchKernelGGL(probe_reg_kernel, dim3(grid), dim3(kRegThreads), 0, s, p);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
