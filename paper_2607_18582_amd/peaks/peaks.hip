// The measured ceilings of mure_peaks.h: a STREAM copy and a register-only
// MFMA loop, each timed with HIP events on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "../../include/mure_peaks.h"

namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

// dst = src over n 16-byte vectors; a block covers 256 U consecutive vectors
// per round (U loads issued before the U stores), rounds grid-strided; NT:
// non-temporal stores (no allocation in the caches for the written lines).
template <int U, bool NT>
__global__ __launch_bounds__(256) void peak_copy_kernel(const v4u* __restrict__ src, v4u* __restrict__ dst,
                                                        int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * 256 * U;
  for (int64_t i = (int64_t)blockIdx.x * 256 * U + threadIdx.x; i < n; i += stride) {
    v4u v[U];
    if (i + (U - 1) * 256 < n) {
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = src[i + u * 256];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if constexpr (NT) __builtin_nontemporal_store(v[u], dst + i + u * 256);
        else dst[i + u * 256] = v[u];
      }
    } else {
      for (int u = 0; u < U && i + u * 256 < n; ++u) dst[i + u * 256] = src[i + u * 256];
    }
  }
}

// Four independent chains of 32x32x16 bf16 MFMAs per wavefront.  Chain q
// multiplies A scaled by 2^-q, so no chain can be merged with another; all
// start at zero and stay small multiples of 2^-20 (the MFMA accumulation is
// not exact in the last bits of larger accumulators: fp32 16x16x4 dropped
// 2^-19 added onto 8), so a lane's sum fixes the number of MFMAs.
__global__ __launch_bounds__(256) void peak_mfma_bf16_kernel(int iters, float* __restrict__ sink) {
  const int tid = threadIdx.x;
  // bf16 2^-8 and 2^-9 (0x3b80, 0x3b00); one less in the exponent field
  // (0x0080 per element) halves a value
  const v4u ab = {0x3b803b80u, 0x3b003b00u, 0x3b803b00u, 0x3b003b80u};
  const v4u half = {0x00800080u, 0x00800080u, 0x00800080u, 0x00800080u};
  const v8bf a0 = __builtin_bit_cast(v8bf, ab);
  const v8bf a1 = __builtin_bit_cast(v8bf, ab - half);
  const v8bf a2 = __builtin_bit_cast(v8bf, ab - 2u * half);
  const v8bf a3 = __builtin_bit_cast(v8bf, ab - 3u * half);
  const v8bf b = __builtin_bit_cast(v8bf, v4u{ab[1], ab[2], ab[3], ab[0]});
  v16f c0, c1, c2, c3;
#pragma unroll
  for (int e = 0; e < 16; ++e) c0[e] = c1[e] = c2[e] = c3[e] = 0.f;
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, b, c3, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 16; ++e) s += c0[e] + c1[e] + c2[e] + c3[e];
  sink[(int64_t)blockIdx.x * 256 + tid] = s;
}

// Eight independent chains of 16x16x4 fp32 MFMAs per wavefront, started at
// (tid + chain) / 1024 in element 0.
__global__ __launch_bounds__(256) void peak_mfma_f32_kernel(int iters, float* __restrict__ sink) {
  const int tid = threadIdx.x;
  const float a = 1.0f / 1024.f, b = 1.0f / 2048.f;
  v4f c[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) c[j] = v4f{(float)(tid + j) * 0x1p-10f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) c[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += c[j][0] + c[j][1] + c[j][2] + c[j][3];
  sink[(int64_t)blockIdx.x * 256 + tid] = s;
}

int hip_status(hipError_t e) { return e == hipSuccess ? 0 : -(int)e; }

// Runs `launch` once untimed and `reps` times timed; *best_ms = the shortest.
template <typename F>
int time_best(hipStream_t s, int reps, F launch, double* best_ms) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) {
    launch();
    e = hipGetLastError();
  }
  double best = 1e300;
  for (int r = 0; r < reps && e == hipSuccess; ++r) {
    e = hipEventRecord(e0, s);
    if (e == hipSuccess) {
      launch();
      e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipEventRecord(e1, s);
    if (e == hipSuccess) e = hipEventSynchronize(e1);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
    if (e == hipSuccess) best = std::min(best, (double)ms);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  *best_ms = best;
  return hip_status(e);
}

}  // namespace

extern "C" int mure_peak_copy(const void* src, void* dst, int64_t bytes, int reps, void* stream, double* gbs) {
  if (!src || !dst || !gbs || bytes <= 0 || bytes % 16 || reps < 1 || reps > 1000) return -1;
  const uintptr_t s0 = (uintptr_t)src, d0 = (uintptr_t)dst;
  if ((s0 | d0) % 16) return -1;
  if (s0 < d0 + (uint64_t)bytes && d0 < s0 + (uint64_t)bytes) return -1;   // overlapping
  const int64_t n = bytes / 16;
  hipStream_t s = (hipStream_t)stream;
  int dev = 0, cus = 256;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_status(e);
  // the best of eight variants: 4 or 8 vectors in flight per thread, plain or
  // non-temporal stores, 8 or 32 blocks per CU (fewer when the copy is small)
  double best = 0.0;
  for (int variant = 0; variant < 8; ++variant) {
    const int u = variant & 1 ? 8 : 4;
    const bool nt = (variant >> 1) & 1;
    const int per_cu = variant & 4 ? 32 : 8;
    const int64_t want = (n + 256 * u - 1) / (256 * u);
    const unsigned grid = (unsigned)std::max<int64_t>(1, std::min<int64_t>(want, (int64_t)cus * per_cu));
    double ms = 0.0;
    const int st = time_best(s, reps, [&] {
      const v4u* sv = (const v4u*)src;
      v4u* dv = (v4u*)dst;
      if (u == 4 && !nt) hipLaunchKernelGGL((peak_copy_kernel<4, false>), dim3(grid), dim3(256), 0, s, sv, dv, n);
      else if (u == 4) hipLaunchKernelGGL((peak_copy_kernel<4, true>), dim3(grid), dim3(256), 0, s, sv, dv, n);
      else if (!nt) hipLaunchKernelGGL((peak_copy_kernel<8, false>), dim3(grid), dim3(256), 0, s, sv, dv, n);
      else hipLaunchKernelGGL((peak_copy_kernel<8, true>), dim3(grid), dim3(256), 0, s, sv, dv, n);
    }, &ms);
    if (st) return st;
    if (ms > 0.0) best = std::max(best, 2.0 * (double)bytes / (ms * 1e-3) / 1e9);
  }
  *gbs = best;
  return 0;
}

extern "C" int mure_peak_mfma(int dtype, int blocks, int iters, int reps, float* sink, void* stream,
                              double* tflops) {
  if ((dtype != 0 && dtype != 1) || blocks < 1 || blocks > 65536 || iters < 1 || iters > 10000000 ||
      reps < 1 || reps > 100 || !sink || !tflops)
    return -1;
  hipStream_t s = (hipStream_t)stream;
  double ms = 0.0;
  const int st = time_best(s, reps, [&] {
    if (dtype == 1)
      hipLaunchKernelGGL(peak_mfma_bf16_kernel, dim3(blocks), dim3(256), 0, s, iters, sink);
    else
      hipLaunchKernelGGL(peak_mfma_f32_kernel, dim3(blocks), dim3(256), 0, s, iters, sink);
  }, &ms);
  if (st) return st;
  // per wavefront and round: 4 x (32x32x16) or 8 x (16x16x4) multiply-adds, 2 flops each
  const double per_round = dtype == 1 ? 4.0 * 32 * 32 * 16 * 2 : 8.0 * 16 * 16 * 4 * 2;
  const double flops = per_round * (double)iters * 4.0 * (double)blocks;
  *tflops = ms > 0.0 ? flops / (ms * 1e-3) / 1e12 : 0.0;
  return 0;
}
