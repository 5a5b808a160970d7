// Self-attention of the chunk's queries over the rolling key/value window
// (current chunk plus the kept past chunks), softmax(q k^T / sqrt(d)) v per
// head, no mask.  Keys of all visible chunks are contiguous rows [0, Lk) of
// the per-head cache, so the kernel sees one key range.
//
// bf16 path (flash-style, one pass over the keys with an online softmax):
//   * workgroup = 4 waves = 128 queries of one head; each wave owns 32 queries
//     whose Q fragments stay in registers for the whole key loop;
//   * per 64-key tile, S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (keys on the
//     MFMA rows, queries on the columns), so each lane holds 32 scores of ONE
//     query: the running max/sum and the output rescale are lane-local except
//     one exchange with the partner lane (lane ^ 32);
//   * O^T += V^T P^T on the same MFMA: the V cache is stored transposed
//     ([d][keys]) so a lane's 8-key operand is one 16-byte LDS read, and the K
//     tile rows are permuted in LDS so that the score registers of each lane
//     are exactly the 8 consecutive keys the P operand needs (no shuffles);
//   * K and V^T tiles are double-buffered in LDS (rows padded by 16 bytes);
//     scores are scaled into the log2 domain by one FMA and exponentiated
//     with exp2; accumulation is float.
// fp32 path: one wave per (query, head), plain online softmax.
#include "xc_internal.h"

#include <math.h>

namespace xc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// MFMA row R of a 32-key M-tile -> key offset within the 64-key tile.
//   R = g*8 + hh*4 + r  ->  key = mt*32 + (g/2)*16 + hh*8 + (g%2)*4 + r
__device__ __forceinline__ int key_of_row(int mt, int R) {
  const int g = R >> 3, hh = (R >> 2) & 1, r = R & 3;
  return mt * 32 + (g >> 1) * 16 + hh * 8 + (g & 1) * 4 + r;
}
// inverse: key offset (0..63) -> LDS row holding it
__device__ __forceinline__ int row_of_key(int key) {
  const int mt = key >> 5, k = key & 31;
  const int g = ((k >> 4) << 1) | ((k >> 2) & 1), hh = (k >> 3) & 1, r = k & 3;
  return mt * 32 + g * 8 + hh * 4 + r;
}

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  The 1-D grid is remapped so that XCD x runs a contiguous range of
// (head, query-tile) items: the query tiles of one head then stream the same
// key/value tiles through one L2 at about the same time.
constexpr int kXcds = 8;

template <int D>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ Kc,
                                                           const bf16* __restrict__ Vt, bf16* __restrict__ O, int L,
                                                           int Mpad, int Lcap, int Lk, int H, int n_qt, float sl2,
                                                           const int* __restrict__ flag) {
  if (flag != nullptr && *flag) return;
  const int total = H * n_qt;
  const int per_xcd = (total + kXcds - 1) / kXcds;
  const int item = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (item >= total) return;
  constexpr int KCH = D / 8;                // 16-byte chunks per key row
  constexpr int KLD = 64 * KCH / 256;       // K chunks staged per thread
  constexpr int VLD = D * 8 / 256;          // V^T chunks staged per thread
  constexpr int DT = D / 32;                // 32-row output tiles (head dims)
  // LDS rows are padded by 16 bytes: the 32 rows a half-wave reads at one
  // chunk position fall in distinct banks, and every fragment address is a
  // per-lane base plus a compile-time offset.
  constexpr int KR = D + 8;                 // K tile row stride (elements)
  constexpr int VR = 64 + 8;                // V^T tile row stride (elements)
  __shared__ __attribute__((aligned(16))) bf16 sK[2][64 * KR];
  __shared__ __attribute__((aligned(16))) bf16 sV[2][D * VR];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hi = lane >> 5, lo = lane & 31;
  const int h = item / n_qt;
  const int q0 = (item - h * n_qt) * 128 + wave * 32;
  const int C = H * D;

  bf16x8 qf[D / 16];
  {
    const bf16* qrow = Q + ((long long)h * Mpad + q0 + lo) * D + hi * 8;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16);
  }
  // per-thread staging sources (advanced by one tile per step) and LDS slots
  const bf16* kg[KLD];
  const bf16* vg[VLD];
  int ks_off[KLD], vs_off[VLD];
#pragma unroll
  for (int i = 0; i < KLD; ++i) {
    const int q = tid + 256 * i, key = q / KCH, c = q % KCH;
    kg[i] = Kc + ((long long)h * Lcap + key) * D + c * 8;
    ks_off[i] = row_of_key(key) * KR + c * 8;
  }
#pragma unroll
  for (int i = 0; i < VLD; ++i) {
    const int q = tid + 256 * i, dd = q >> 3, c = q & 7;
    vg[i] = Vt + ((long long)h * D + dd) * Lcap + c * 8;
    vs_off[i] = dd * VR + c * 8;
  }
  const int k_frag = lo * KR + hi * 8;   // + mt*32*KR + ks*16
  const int v_frag = lo * VR + hi * 8;   // + dt*32*VR + kv*16

  f32x16 oacc[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float lazy = 8.0f / sl2;

  u32x4 rk[KLD], rv[VLD];
  auto gload = [&](int j) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < KLD; ++i) rk[i] = *reinterpret_cast<const u32x4*>(kg[i] + (long long)j * 64 * D);
#pragma unroll
    for (int i = 0; i < VLD; ++i) rv[i] = *reinterpret_cast<const u32x4*>(vg[i] + j * 64);
  };
  auto sstore = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < KLD; ++i) *reinterpret_cast<u32x4*>(&sK[buf][ks_off[i]]) = rk[i];
#pragma unroll
    for (int i = 0; i < VLD; ++i) *reinterpret_cast<u32x4*>(&sV[buf][vs_off[i]]) = rv[i];
  };

  const int NT = (Lk + 63) / 64;
  auto step = [&](int j, int cur) __attribute__((always_inline)) {
    if (j + 1 < NT) gload(j + 1);
    f32x16 sacc[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[mt][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sK[cur][k_frag + mt * 32 * KR + ks * 16]);
        sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sacc[mt], 0, 0, 0);
      }
    }
    // running max in raw score units; p = 2^(s*c - m*c) with c = log2(e)/sqrt(d).
    // The rescale of the output accumulators is skipped while the max has
    // grown by less than 8/c since the last rescale (p then stays <= 2^8,
    // harmless for the float sums and the bf16 probabilities).
    if ((j + 1) * 64 > Lk) {  // last tile: mask keys past the window
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = j * 64 + key_of_row(mt, (i >> 2) * 8 + hi * 4 + (i & 3));
          if (key >= Lk) sacc[mt][i] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[mt][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    if (mx > m_run + lazy) {
      const float m_new = fmaxf(mx, m_run);
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * sl2);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
      m_run = m_new;
    }
    const float msc = -m_run * sl2;
    float ps = 0.f;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[mt][i], sl2, msc));
        sacc[mt][i] = p;
        ps += p;
      }
    l_run += ps;
    bf16x8 pb[4];
#pragma unroll
    for (int kv = 0; kv < 4; ++kv)
#pragma unroll
      for (int i = 0; i < 8; ++i) pb[kv][i] = (bf16)sacc[kv >> 1][(kv & 1) * 8 + i];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int kv = 0; kv < 4; ++kv) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sV[cur][v_frag + dt * 32 * VR + kv * 16]);
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[kv], oacc[dt], 0, 0, 0);
      }
    if (j + 1 < NT) sstore(cur ^ 1);
    __syncthreads();
  };

  gload(0);
  sstore(0);
  __syncthreads();
  for (int j = 0; j < NT; j += 2) {
    step(j, 0);
    if (j + 1 < NT) step(j + 1, 1);
  }
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  const int q = q0 + lo;
  if (q < L) {
    bf16* orow = O + (long long)q * C + h * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int dd = dt * 32 + g * 8 + hi * 4;
        typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
        bf16x4 o4;
#pragma unroll
        for (int r = 0; r < 4; ++r) o4[r] = (bf16)(oacc[dt][g * 4 + r] * inv);
        *reinterpret_cast<bf16x4*>(orow + dd) = o4;
      }
  }
}

__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ Q, const float* __restrict__ Kc,
                                                      const float* __restrict__ Vt, float* __restrict__ O, int L,
                                                      int Mpad, int Lcap, int Lk, int H, int D, float scale,
                                                      const int* __restrict__ flag) {
  if (flag != nullptr && *flag) return;
  __shared__ float sq[128];
  __shared__ float sp[64];
  const int lane = threadIdx.x, q = blockIdx.x, h = blockIdx.y;
  for (int i = lane; i < D; i += 64) sq[i] = Q[((long long)h * Mpad + q) * D + i];
  __syncthreads();
  const float* Kh = Kc + (long long)h * Lcap * D;
  const float* Vh = Vt + (long long)h * D * Lcap;
  float m = -INFINITY, l = 0.f, o0 = 0.f, o1 = 0.f;
  for (int k0 = 0; k0 < Lk; k0 += 64) {
    const int key = k0 + lane;
    float s = -INFINITY;
    if (key < Lk) {
      float acc = 0.f;
      for (int i = 0; i < D; ++i) acc += sq[i] * Kh[(long long)key * D + i];
      s = acc * scale;
    }
    float mx = s;
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    const float m_new = fmaxf(m, mx);
    const float alpha = expf(m - m_new);
    const float p = key < Lk ? expf(s - m_new) : 0.f;
    float ps = p;
    for (int off = 32; off > 0; off >>= 1) ps += __shfl_xor(ps, off, 64);
    l = l * alpha + ps;
    o0 *= alpha;
    o1 *= alpha;
    sp[lane] = p;
    __syncthreads();
    const int nk = min(64, Lk - k0);
    for (int jj = 0; jj < nk; ++jj) {
      if (lane < D) o0 += sp[jj] * Vh[(long long)lane * Lcap + k0 + jj];
      if (lane + 64 < D) o1 += sp[jj] * Vh[(long long)(lane + 64) * Lcap + k0 + jj];
    }
    __syncthreads();
    m = m_new;
  }
  float* orow = O + (long long)q * H * D + h * D;
  if (lane < D) orow[lane] = o0 / l;
  if (lane + 64 < D) orow[lane + 64] = o1 / l;
}

}  // namespace

// bf16 requirements (checked by the caller): D in {64, 128}; Q has Mpad >=
// roundup(L, 128) rows per head; the caches have Lcap >= roundup(Lk, 64) rows.
void launch_attention(int dtype, const void* q, const void* kc, const void* vt, void* o, int L, int Mpad, int Lcap,
                      int Lk, int H, int D, const int* flag, hipStream_t st) {
  if (dtype == 1) {
    const int n_qt = (L + 127) / 128;
    const int per_xcd = (H * n_qt + kXcds - 1) / kXcds;
    const dim3 grid(per_xcd * kXcds);
    const float sl2 = 1.4426950408889634f / sqrtf((float)D);
    if (D == 128)
      attn_bf16_kernel<128><<<grid, 256, 0, st>>>((const bf16*)q, (const bf16*)kc, (const bf16*)vt, (bf16*)o, L,
                                                  Mpad, Lcap, Lk, H, n_qt, sl2, flag);
    else
      attn_bf16_kernel<64><<<grid, 256, 0, st>>>((const bf16*)q, (const bf16*)kc, (const bf16*)vt, (bf16*)o, L,
                                                 Mpad, Lcap, Lk, H, n_qt, sl2, flag);
  } else {
    dim3 grid(L, H);
    attn_f32_kernel<<<grid, 64, 0, st>>>((const float*)q, (const float*)kc, (const float*)vt, (float*)o, L, Mpad,
                                         Lcap, Lk, H, D, 1.0f / sqrtf((float)D), flag);
  }
}

}  // namespace xc
