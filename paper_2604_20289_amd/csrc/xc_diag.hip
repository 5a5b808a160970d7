// Measurement aid (not a step of the method): the bf16 MFMA rate the chip
// sustains on a loop that keeps every operand in registers, i.e. the
// practical ceiling the contractions of the block can be compared with.
//
// Each wave repeats independent MFMA chains on operands it filled once: 4
// chains of 32x32x16 or 16 chains of 16x16x32 (measured: with 4 waves per
// SIMD the 32x32x16 rate is flat from 1 chain up, the 16x16x32 rate needs
// 12 or more), so the matrix pipe never waits on an accumulator.  The
// operands matter: the matrix cores draw power in proportion to the bits that
// toggle, and the clock the chip holds under that load follows, so the rate
// is measured both on random bf16 operands (the case of real activations and
// weights) and on zeros.
#include "xc_internal.h"

#include <stdint.h>

namespace xc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kDiagThreads = 256;
constexpr int kDiagGroups = 1024;  // four waves per SIMD on 256 CUs

__device__ __forceinline__ uint32_t xorshift(uint32_t x) {
  x ^= x << 13;
  x ^= x >> 17;
  x ^= x << 5;
  return x;
}

// a bf16 in [-2, -0.5] U [0.5, 2) with a random mantissa, or 0
__device__ __forceinline__ __bf16 operand(uint32_t& x, int random) {
  x = xorshift(x);
  const uint32_t bits = random ? ((x & 1u) << 15) | ((126u + ((x >> 1) & 1u)) << 7) | ((x >> 2) & 0x7fu) : 0u;
  return __builtin_bit_cast(__bf16, (unsigned short)bits);
}

template <int SHAPE>
__global__ __launch_bounds__(kDiagThreads) void mfma_loop_kernel(int iters, int random, uint32_t seed) {
  uint32_t x = seed ^ ((blockIdx.x * kDiagThreads + threadIdx.x + 1u) * 0x9E3779B9u);
  bf16x8 a[2], b[2];
#pragma unroll
  for (int k = 0; k < 2; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[k][e] = operand(x, random);
      b[k][e] = operand(x, random);
    }
  float s = 0.f;
  if constexpr (SHAPE == 0) {
    f32x16 acc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
    for (int it = 0; it < iters; ++it)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[c & 1], b[c & 1], acc[c], 0, 0, 0);
#pragma unroll
    for (int c = 0; c < 4; ++c) s += acc[c][0];
  } else {
    f32x4 acc[16];
#pragma unroll
    for (int c = 0; c < 16; ++c)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[c][r] = 0.f;
    for (int it = 0; it < iters / 2; ++it)
#pragma unroll
      for (int c = 0; c < 16; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[c & 1], b[c & 1], acc[c], 0, 0, 0);
#pragma unroll
    for (int c = 0; c < 16; ++c) s += acc[c][0];
  }
  // the accumulators are consumed by an (empty) asm statement: the loop stays
  asm volatile("; mfma loop result %0" ::"v"(s));
}

}  // namespace

// Flops per wave and iteration: 4 x 32x32x16 products, or 16 x 16x16x32
// products every second iteration: 131072 either way.  One untimed launch
// lets the clocks settle under the load; the best of three timed launches
// (about 8 ms each) is reported.
hipError_t mfma_rate(int shape, int random, hipStream_t st, double* tflops) {
  constexpr int kIters = 15000;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t err = hipEventCreate(&e0);
  if (err == hipSuccess) err = hipEventCreate(&e1);
  auto launch = [&](int iters) {
    if (shape == 0)
      mfma_loop_kernel<0><<<kDiagGroups, kDiagThreads, 0, st>>>(iters, random, 12345u);
    else
      mfma_loop_kernel<1><<<kDiagGroups, kDiagThreads, 0, st>>>(iters, random, 12345u);
    return hipGetLastError();
  };
  float ms = 0.f;
  if (err == hipSuccess) err = launch(kIters);
  for (int rep = 0; rep < 3 && err == hipSuccess; ++rep) {
    float t = 0.f;
    err = hipEventRecord(e0, st);
    if (err == hipSuccess) err = launch(kIters);
    if (err == hipSuccess) err = hipEventRecord(e1, st);
    if (err == hipSuccess) err = hipEventSynchronize(e1);
    if (err == hipSuccess) err = hipEventElapsedTime(&t, e0, e1);
    if (err == hipSuccess && (ms == 0.f || t < ms)) ms = t;
  }
  if (e0 != nullptr) (void)hipEventDestroy(e0);
  if (e1 != nullptr) (void)hipEventDestroy(e1);
  if (err != hipSuccess) return err;
  const double flops = (double)kDiagGroups * (kDiagThreads / 64) * kIters * 131072.0;
  *tflops = ms > 0.f ? flops / (ms * 1e-3) / 1e12 : 0.0;
  return hipSuccess;
}

}  // namespace xc
