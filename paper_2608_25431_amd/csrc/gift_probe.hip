// LDS read-rate and VALU issue-rate probes for the benchmark's LDS and VALU
// ceilings of the seal kernel.
//
// The seal kernel's per-block work is bound by two kinds of LDS reads: random
// 4-byte T-table lookups (each lane in its own copy of the table, so a wave's
// lookups never meet in a bank) and 16-byte reads of nibble-indexed GHASH
// tables (a 256-byte sub-table spans every bank once, so lanes either share
// an entry or use disjoint banks).  These kernels issue only such reads, at
// fixed per-lane addresses of the same forms, as fast as the LDS accepts
// them: batches of 15 independent reads (the most the LDS counter tracks)
// with one wait per batch and no other arithmetic, on one 1024-thread
// workgroup per CU with the LDS allocation of the seal kernel.  The shader
// clock counts the batches' time; the reference clock beside it gives the
// clock rate.  The VALU probes (k_valu) issue the kernel's two most common
// vector instructions the same way.
//
// Built into libgift_probe.so, apart from the library: only the benchmark
// loads it.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 1024;
constexpr int kBatch = 15;             // LDS reads in flight per wave
constexpr int kMixed32 = 13;           // mixed batch: 13 four-byte and 2 sixteen-byte reads
constexpr uint32_t kT32Bytes = 65536;  // two 1 KiB tables x 32 copies: the seal kernel's AES region
constexpr uint32_t kT128Bytes = 8192;  // 32 nibble positions x 16 entries x 16 B: one GHASH table set
constexpr uint32_t kLdsBytes = 160u * 1024u - 64u;  // one workgroup per CU, as in the seal kernel

typedef __attribute__((address_space(3))) uint8_t lds_byte;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// mode 0: kBatch 4-byte reads per step at (byte << 8) | 4 * (lane mod 32) |
// table bit, the seal kernel's T-table form; mode 1: kBatch 16-byte reads
// per step at 256 * sub-table + 16 * nibble; mode 2: kMixed32 of the first
// kind and kBatch - kMixed32 of the second per step.
template <int MODE>
__global__ __launch_bounds__(kThreads) void k_probe(uint32_t steps, uint32_t* sink, unsigned long long* stamps) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const uint32_t tid = threadIdx.x;
  for (uint32_t i = tid; i < (kT32Bytes + kT128Bytes) / 4u; i += kThreads) ((uint32_t*)smem)[i] = i * 2654435761u;
  if (tid == 0) smem[kLdsBytes - 1u - (blockIdx.x & 63u)] = 1;  // keeps the whole allocation
  __syncthreads();
  const uint32_t base = (uint32_t)(uintptr_t)(lds_byte*)smem;
  uint32_t addr[kBatch];
#pragma unroll
  for (int k = 0; k < kBatch; k++) {
    const uint32_t h = (tid * 7919u + (uint32_t)k * 104729u + blockIdx.x * 31u) * 2654435761u;
    const bool wide = MODE == 1 || (MODE == 2 && k >= kMixed32);
    addr[k] = wide ? base + kT32Bytes + ((((uint32_t)k * 5u + (tid >> 6)) & 31u) << 8) + (((h >> 20) & 15u) << 4)
                   : base + (((h >> 24) << 8) | ((tid & 31u) << 2) | (((uint32_t)k & 1u) << 7));
  }
  uint32_t acc = 0;
  __syncthreads();
  const unsigned long long c0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (uint32_t s = 0; s < steps; s++) {
    uint32_t v[kBatch];
    u32x4 w[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; k++) {
      if (MODE == 1 || (MODE == 2 && k >= kMixed32))
        asm volatile("ds_read_b128 %0, %1" : "=v"(w[k]) : "v"(addr[k]));
      else
        asm volatile("ds_read_b32 %0, %1" : "=v"(v[k]) : "v"(addr[k]));
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    // ties every result to a point after the wait
#pragma unroll
    for (int k = 0; k < kBatch; k++) {
      if (MODE == 1 || (MODE == 2 && k >= kMixed32))
        asm volatile("" : "+v"(w[k]));
      else
        asm volatile("" : "+v"(v[k]));
    }
    acc ^= (MODE == 1) ? w[0].x : v[0];
  }
  __syncthreads();
  const unsigned long long c1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  sink[blockIdx.x * kThreads + tid] = acc;
  if (tid == 0) {
    stamps[2 * blockIdx.x] = c1 - c0;
    stamps[2 * blockIdx.x + 1] = r1 - r0;
  }
}

// Vector-ALU rate of the seal kernel's two most common instructions: eight
// accumulators per thread, each step one v_bitop3_b32 (OP 0) or one
// v_perm_b32 (OP 1) per accumulator on its own and other accumulators'
// values (the byte selectors stay fixed), so a wave always has independent
// instructions to issue.  It holds the seal kernel's LDS allocation, so that
// it too runs one workgroup per CU.
template <int OP>
__global__ __launch_bounds__(kThreads) void k_valu(uint32_t steps, uint32_t* sink, unsigned long long* stamps) {
  __shared__ uint8_t smem[kLdsBytes];
  if (threadIdx.x == 0) smem[kLdsBytes - 1u - (blockIdx.x & 63u)] = 1;
  uint32_t a[8], sel[8];
#pragma unroll
  for (int k = 0; k < 8; k++) {
    a[k] = (threadIdx.x + 1u) * (2654435761u + 40503u * (uint32_t)k);
    sel[k] = ((threadIdx.x + (uint32_t)k) * 0x01030507u) & 0x07070707u;  // byte selectors 0-7
  }
  __syncthreads();
  const unsigned long long c0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (uint32_t s = 0; s < steps; s++) {
#pragma unroll
    for (int k = 0; k < 8; k++) {
      if (OP == 0)
        a[k] = __builtin_amdgcn_bitop3_b32(a[k], a[(k + 1) & 7], a[(k + 3) & 7], 0x96);
      else
        a[k] = __builtin_amdgcn_perm(a[k], a[(k + 1) & 7], sel[k]);
    }
  }
  __syncthreads();
  const unsigned long long c1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  uint32_t acc = 0;
#pragma unroll
  for (int k = 0; k < 8; k++) acc ^= a[k];
  if (threadIdx.x == 0) acc ^= smem[kLdsBytes - 1u - (blockIdx.x & 63u)];
  sink[blockIdx.x * kThreads + threadIdx.x] = acc;
  if (threadIdx.x == 0) {
    stamps[2 * blockIdx.x] = c1 - c0;
    stamps[2 * blockIdx.x + 1] = r1 - r0;
  }
}

}  // namespace

extern "C" {

// Runs probe `mode` on `cus` workgroups of `steps` steps, once to warm up and
// once timed, and returns in *clk_per_step the mean shader clocks per step
// of one workgroup (1024 threads) and in *mhz the shader clock rate over the
// same interval (shader clocks against the 100 MHz reference clock).  Modes
// 0-2 are the LDS probes (kBatch reads per thread and step, as above); 3 and
// 4 the VALU probes (8 v_bitop3_b32 or 8 v_perm_b32 per thread and step).
// Synchronous on the null stream; allocates and frees its own buffers.
// Returns a hipError_t (hipErrorInvalidValue for a bad mode, zero counts or
// null pointers).
int gift_probe_lds(uint32_t mode, uint32_t cus, uint32_t steps, double* clk_per_step, double* mhz) {
  if (mode > 4 || cus == 0 || steps == 0 || !clk_per_step || !mhz) return (int)hipErrorInvalidValue;
  uint32_t* sink = nullptr;
  unsigned long long* st = nullptr;
  hipError_t e = hipMalloc((void**)&sink, sizeof(uint32_t) * kThreads * cus);
  if (e == hipSuccess) e = hipMalloc((void**)&st, sizeof(unsigned long long) * 2 * cus);
  for (int rep = 0; rep < 2 && e == hipSuccess; rep++) {
    if (mode == 0) hipLaunchKernelGGL(k_probe<0>, dim3(cus), dim3(kThreads), 0, 0, steps, sink, st);
    if (mode == 1) hipLaunchKernelGGL(k_probe<1>, dim3(cus), dim3(kThreads), 0, 0, steps, sink, st);
    if (mode == 2) hipLaunchKernelGGL(k_probe<2>, dim3(cus), dim3(kThreads), 0, 0, steps, sink, st);
    if (mode == 3) hipLaunchKernelGGL(k_valu<0>, dim3(cus), dim3(kThreads), 0, 0, steps, sink, st);
    if (mode == 4) hipLaunchKernelGGL(k_valu<1>, dim3(cus), dim3(kThreads), 0, 0, steps, sink, st);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess) {
    unsigned long long* h = new unsigned long long[2 * cus];
    e = hipMemcpy(h, st, sizeof(unsigned long long) * 2 * cus, hipMemcpyDeviceToHost);
    double ck = 0, rt = 0;
    for (uint32_t i = 0; i < cus; i++) {
      ck += (double)h[2 * i];
      rt += (double)h[2 * i + 1];
    }
    delete[] h;
    if (e == hipSuccess) {
      *clk_per_step = ck / cus / steps;
      *mhz = rt > 0 ? 100.0 * ck / rt : 0.0;
    }
  }
  if (sink) (void)hipFree(sink);
  if (st) (void)hipFree(st);
  return (int)e;
}

}  // extern "C"
