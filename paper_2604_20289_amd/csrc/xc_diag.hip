// Measurement aids (not steps of the method): the bf16 MFMA rate the chip
// sustains on a loop that keeps every operand in registers, i.e. the
// practical ceiling the contractions of the block can be compared with; and
// the rate of the global -> LDS request stream the GEMMs stage their operands
// with, as a function of the row segment one request fetches; and the MFMA
// rate under the attention loop's instruction mix (its LDS operand reads and
// its softmax VALU work) on data that depends on nothing, i.e. what that mix
// allows before any dependency or synchronisation is paid.
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

// Instruction mixes of the attention loop at its occupancy (one 512-thread
// workgroup per CU, two waves per SIMD; the 96 KB of LDS keep a second
// workgroup off the CU).  Per wave and iteration: 32 MFMAs 32x32x16 on 4
// chains with the B operand in registers and the A operand one of 8
// fragment registers, which MIX bit 0 refills from LDS after each use (one
// 16-byte read per MFMA, used 8 MFMAs later, from one of two 32 KB halves
// by iteration: the attention kernel's K and V^T operand traffic); MIX bit 1 adds the VALU work a 64-key tile's softmax
// costs a wave there: per lane the max of its 32 scores, 32 fused
// scale-and-subtract, 32 exp2, 16 bf16 pair conversions and 16 two-wide dot
// products for the row sum.  The probabilities become the next iteration's
// scores, so nothing is loop-invariant and no extra instruction is needed.
constexpr int kMixGroups = 256;
constexpr int kMixThreads = 512;

template <int MIX>
__global__ __launch_bounds__(512, 1) void mfma_mix_kernel(int iters, int random, uint32_t seed) {
  __shared__ __attribute__((aligned(1024))) __bf16 lds[48 * 1024];  // 96 KB; 64 fragment rows of 1 KB used
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  const int tid = threadIdx.x, lane = tid & 63;
  uint32_t x = seed ^ ((blockIdx.x * kMixThreads + tid + 1u) * 0x9E3779B9u);
  for (int i = tid; i < 64 * 512; i += kMixThreads) lds[i] = operand(x, random);
  __syncthreads();
  bf16x8 b, f[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = operand(x, random);
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = *reinterpret_cast<const bf16x8*>(lds + j * 512 + lane * 8);
  f32x16 acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  float sc[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) sc[i] = (float)((x >> (i & 15)) & 255) * (1.0f / 256.0f);
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float m = 0.f, l = 0.f;
  for (int it = 0; it < iters; ++it) {
    const __bf16* half = lds + (it & 1) * 32 * 512 + lane * 8;  // the reads' offsets are immediates
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      acc[j & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[j & 7], b, acc[j & 3], 0, 0, 0);
      if constexpr ((MIX & 1) != 0)
        f[j & 7] = *reinterpret_cast<const bf16x8*>(half + j * 512);
    }
    if constexpr ((MIX & 2) != 0) {
      float mx = m;
#pragma unroll
      for (int i = 0; i < 32; ++i) mx = fmaxf(mx, sc[i]);
#pragma unroll
      for (int i = 0; i < 32; ++i) sc[i] = __builtin_amdgcn_exp2f(fmaf(sc[i], 0.0884f, -mx));
#pragma unroll
      for (int i = 0; i < 32; i += 2) {
        const f32x2 pf = {sc[i], sc[i + 1]};
        l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_convertvector(pf, bf16x2), ones, l, false);
      }
      m = mx;
    }
  }
  float t = l + m;
#pragma unroll
  for (int c = 0; c < 4; ++c) t += acc[c][0];
  asm volatile("; mfma mix result %0" ::"v"(t));
}

// global -> LDS request stream: a workgroup streams tile t's rows (shared
// with the other tiles of its row block, like the M-tiles of a GEMM) through
// a 3-slot ring of 24 KB stages, two stages ahead, one barrier per stage and
// no arithmetic; each stage takes RB bytes of every one of its 24 KB / RB
// rows (RB = 64, 128 or 256: the row segment one request fetches).
constexpr int kDmaGroups = 1008;
constexpr int kDmaBlocks = 28;          // row blocks of 384 x 64-byte-stage rows shared by the tiles
constexpr int kDmaRowElems = 1536;      // bf16 elements per matrix row

__device__ __forceinline__ void dma16(const __bf16* src, __bf16* lds_block) {
  __builtin_amdgcn_global_load_lds(src, lds_block, 16, 0, 0);
}

template <int RB>
__global__ __launch_bounds__(256, 2) void dma_stream_kernel(const __bf16* __restrict__ A) {
  __shared__ __attribute__((aligned(1024))) __bf16 lds[3][12 * 1024];
  constexpr int CPR = RB / 16;                 // 16-byte chunks per row segment
  constexpr int RPI = 64 / CPR;                // rows per 1 KB request
  constexpr int ROWS = 24 * RPI;               // rows per stage
  constexpr int STAGES = kDmaRowElems * 2 / RB;  // one pass over the rows
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const __bf16* base = A + (long long)(blockIdx.x % (kDmaBlocks * 384 / ROWS)) * ROWS * kDmaRowElems;
  auto issue = [&](int st, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      const int I = wave + 4 * i;
      const int row = I * RPI + lane / CPR, c = lane % CPR;
      dma16(base + (long long)row * kDmaRowElems + st * (RB / 2) + c * 8, &lds[buf][I * 512]);
    }
  };
#define XC_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((0x3f70) | ((n) & 15) | (((n) >> 4) << 14))
  issue(0, 0);
  issue(1, 1);
  XC_WAIT_VMCNT(6);
  __syncthreads();
  for (int st = 0; st < STAGES; ++st) {
    issue(min(st + 2, STAGES - 1), (st + 2) % 3);
    XC_WAIT_VMCNT(6);
    __syncthreads();
  }
  XC_WAIT_VMCNT(0);
#undef XC_WAIT_VMCNT
}

}  // namespace

hipError_t lds_dma_rate(int row_bytes, hipStream_t st, double* tbps) {
  const size_t elems = (size_t)kDmaBlocks * 384 * kDmaRowElems;
  __bf16* A = nullptr;
  hipError_t err = hipMalloc(&A, elems * sizeof(__bf16));
  if (err != hipSuccess) return err;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  err = hipMemsetAsync(A, 0, elems * sizeof(__bf16), st);
  if (err == hipSuccess) err = hipEventCreate(&e0);
  if (err == hipSuccess) err = hipEventCreate(&e1);
  auto launch = [&]() {
    if (row_bytes == 64)
      dma_stream_kernel<64><<<kDmaGroups, 256, 0, st>>>(A);
    else if (row_bytes == 128)
      dma_stream_kernel<128><<<kDmaGroups, 256, 0, st>>>(A);
    else
      dma_stream_kernel<256><<<kDmaGroups, 256, 0, st>>>(A);
    return hipGetLastError();
  };
  float ms = 0.f;
  for (int rep = 0; rep < 3 && err == hipSuccess; ++rep) err = launch();
  for (int rep = 0; rep < 5 && err == hipSuccess; ++rep) {
    float t = 0.f;
    err = hipEventRecord(e0, st);
    if (err == hipSuccess) err = launch();
    if (err == hipSuccess) err = hipEventRecord(e1, st);
    if (err == hipSuccess) err = hipEventSynchronize(e1);
    if (err == hipSuccess) err = hipEventElapsedTime(&t, e0, e1);
    if (err == hipSuccess && (ms == 0.f || t < ms)) ms = t;
  }
  if (e0 != nullptr) (void)hipEventDestroy(e0);
  if (e1 != nullptr) (void)hipEventDestroy(e1);
  const hipError_t ferr = hipStreamSynchronize(st);
  (void)hipFree(A);
  if (err != hipSuccess) return err;
  if (ferr != hipSuccess) return ferr;
  // every tile moves all 24 KB stages of one pass over its rows
  const double bytes = (double)kDmaGroups * (kDmaRowElems * 2 / row_bytes) * 24.0 * 1024.0;
  *tbps = ms > 0.f ? bytes / (ms * 1e-3) / 1e12 : 0.0;
  return hipSuccess;
}

// Flops per wave and iteration: 4 x 32x32x16 products, or 16 x 16x16x32
// products every second iteration: 131072 either way (shapes 0, 1); 32 x
// 32x32x16 products = 1048576 for the mixes (shapes 2-4).  One untimed
// launch lets the clocks settle under the load; the best of three timed
// launches (about 8 ms each for shapes 0 and 1) is reported.
hipError_t mfma_rate(int shape, int random, hipStream_t st, double* tflops) {
  constexpr int kIters = 15000, kMixIters = 4000;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t err = hipEventCreate(&e0);
  if (err == hipSuccess) err = hipEventCreate(&e1);
  auto launch = [&](int iters) {
    switch (shape) {
      case 0: mfma_loop_kernel<0><<<kDiagGroups, kDiagThreads, 0, st>>>(iters, random, 12345u); break;
      case 1: mfma_loop_kernel<1><<<kDiagGroups, kDiagThreads, 0, st>>>(iters, random, 12345u); break;
      case 2: mfma_mix_kernel<1><<<kMixGroups, kMixThreads, 0, st>>>(kMixIters, random, 12345u); break;
      case 3: mfma_mix_kernel<2><<<kMixGroups, kMixThreads, 0, st>>>(kMixIters, random, 12345u); break;
      default: mfma_mix_kernel<3><<<kMixGroups, kMixThreads, 0, st>>>(kMixIters, random, 12345u); break;
    }
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
  const double flops = shape < 2 ? (double)kDiagGroups * (kDiagThreads / 64) * kIters * 131072.0
                                 : (double)kMixGroups * (kMixThreads / 64) * kMixIters * 1048576.0;
  *tflops = ms > 0.f ? flops / (ms * 1e-3) / 1e12 : 0.0;
  return hipSuccess;
}

}  // namespace xc
