// Dense projections of the DiT block: C[M][N] = A[M][K] * W[N][K]^T with fused
// epilogues (bias, gated residual, tanh-GELU, cached-residual store, and for
// the QKV projection the per-head RMSNorm with the K / V^T cache stores).
//
// bf16 path, two kernels built on v_mfma_f32_32x32x16_bf16 with float
// accumulation.  Both operands are K-contiguous (activations row-major,
// weights [out][in]), so a lane's MFMA operand is one 16-byte LDS read, and
// stage tiles go from global memory straight into LDS (global_load_lds).
//  * gemm_bf16_wide: one 8-wave workgroup per CU, 256 x 256 tiles (QKV,
//    MLP up) or 256 x 192 tiles (output and MLP-down projections), 64-deep
//    stages;
//  * gemm_bf16_kernel: (64*MT) x 128 tiles, two workgroups per CU, 32-deep
//    stages; widths the wide tiles do not divide.
// Both run the element-wise epilogues through tile_epilogue (software-
// pipelined operand loads, range-checked buffer stores) and the QKV epilogue
// through qkv_epilogue.
//
// fp32 path: a plain LDS-tiled FMA GEMM (64x64 tiles, 4x4 per thread) used
// for float32 models.
#include "xc_internal.h"

#include <math.h>

namespace xc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// tanh-approximated GELU, 0.5 v (1 + tanh(u)) with u = sqrt(2/pi) (v + 0.044715 v^3),
// evaluated through the identity 0.5 (1 + tanh(u)) = 1 / (1 + e^(-2u)):
// v / (1 + 2^z), z = -2 log2(e) u, on the hardware exp2 and reciprocal.  For
// v -> -inf, 2^z -> inf and the result -> -0; no branch, no NaN for finite v.
__device__ __forceinline__ float gelu_tanh(float v) {
  constexpr float c1 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  constexpr float c3 = c1 * 0.044715f;
  const float z = v * fmaf(c3, v * v, c1);
  return v * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}

template <typename T>
__device__ __forceinline__ T cvt(float v);
template <>
__device__ __forceinline__ float cvt<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16 cvt<bf16>(float v) { return (bf16)v; }

template <int MODE, typename T>
__device__ __forceinline__ void epilogue(const EpiArgs& e, int m, int n, float acc) {
  const long long i = (long long)m * e.N + n;
  const float v = acc + e.bias[n];
  if constexpr (MODE == EPI_BIAS_F32) {
    e.out_f32[i] = v;
  } else if constexpr (MODE == EPI_OPROJ) {
    e.out_f32[i] = e.resid[i] + e.gate[n] * v;
  } else if constexpr (MODE == EPI_UP) {
    reinterpret_cast<T*>(e.out_t)[i] = cvt<T>(gelu_tanh(v));
  } else if constexpr (MODE == EPI_DOWN) {
    const float xin = e.xin[i];
    const float y = e.resid[i] + e.gate[n] * v;
    e.out_f32[i] = y;
    if (e.out_t != nullptr) reinterpret_cast<T*>(e.out_t)[i] = cvt<T>(y - xin);
  }
}

// Element-wise epilogue of an MT x NT block of 32x32 accumulators (both bf16
// GEMM kernels).  The lane's rows are m0 + r0 + mt*32 + g*8 + r (m0 the tile's
// first row, BM its height), its columns cb + nt*32.  Column constants
// (bias, gate) are read once.  The 16 blocks of 4 rows are processed one at
// a time (which bounds the live registers) and software-pipelined: the
// operand loads of block k+1 (residual, block input) are issued before block
// k is computed and stored, so the HBM latency of one block overlaps the
// work of the previous one instead of being paid 16 times in a row.  Stores
// go through buffer descriptors whose range ends at row M (a store past it is
// dropped by the hardware), so no branch separates them: the compiler then
// knows how many stores follow each load batch and waits only for the loads
// it needs, not for every earlier store.  Loads of rows past M use a clamped
// row.  EPI_DOWN with csum_part: each 32-row block's per-camera column sums of
// y and of the stored residual (two slots: the camera of the block's first
// token, the next camera from token rb_split on) are summed in registers
// over the lane's rows, combined with the partner half-wave and written, one
// slot per half-wave (a zero-length range when off).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(void* base, long long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, (int)bytes, 0x00020000);
}

template <int MODE, int MT, int NT>
__device__ __forceinline__ void tile_epilogue(const EpiArgs& e, const f32x16 (&acc)[MT][NT], int m0, int r0, int cb,
                                              int M, int BM) {
  constexpr bool kRes = MODE == EPI_OPROJ || MODE == EPI_DOWN;
  constexpr bool kXin = MODE == EPI_DOWN;
  // the tile's rows [m0, min(m0 + BM, M)) of every output, as buffer ranges
  const long long rows = min(BM, M - m0);
  const __amdgpu_buffer_rsrc_t out_f = tile_rsrc(e.out_f32 + (long long)m0 * e.N, rows * e.N * 4);
  const __amdgpu_buffer_rsrc_t out_b =
      tile_rsrc(reinterpret_cast<bf16*>(e.out_t) + (long long)m0 * e.N, e.out_t != nullptr ? rows * e.N * 2 : 0);
  float bias[NT], gate[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    bias[nt] = e.bias[cb + nt * 32];
    gate[nt] = kRes ? e.gate[cb + nt * 32] : 0.f;
  }
  const long long N = e.N;
  // column-sum partials (EPI_DOWN): per kind one range of n_rb x 2 x N floats
  const bool csum = kXin && e.csum_part != nullptr;
  const long long part_bytes = csum ? (long long)e.n_rb * 2 * N * 4 : 0;
  const __amdgpu_buffer_rsrc_t part_y = tile_rsrc(e.csum_part, part_bytes);
  const __amdgpu_buffer_rsrc_t part_d = tile_rsrc(e.csum_part + (csum ? (long long)e.n_rb * 2 * N : 0), part_bytes);
  const int rb0 = (m0 + (r0 & ~31)) >> 5, roff = r0 & 31;  // the lane's first 32-row block, its offset in it
  int split[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) split[mt] = csum ? e.rb_split[min(rb0 + mt, e.n_rb - 1)] : 32;
  float sy[2][NT], sd[2][NT];
  float res[2][4][NT], xin[2][4][NT];
  auto load = [&](int blk, int slot) __attribute__((always_inline)) {
    const int mt = blk >> 2, g = blk & 3;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const long long il = (long long)min(m0 + r0 + mt * 32 + g * 8 + r, M - 1) * N + cb;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        if constexpr (kRes) res[slot][r][nt] = e.resid[il + nt * 32];
        if constexpr (kXin) xin[slot][r][nt] = e.xin[il + nt * 32];
      }
    }
  };
  load(0, 0);
#pragma unroll
  for (int blk = 0; blk < 4 * MT; ++blk) {
    const int mt = blk >> 2, g = blk & 3, slot = blk & 1;
    if (blk + 1 < 4 * MT) load(blk + 1, slot ^ 1);
    __builtin_amdgcn_sched_barrier(0);
    // this block's 4 x NT accumulators move to VGPRs here, not all at once
    float v[4][NT];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        v[r][nt] = acc[mt][nt][g * 4 + r];
        asm volatile("" : "+v"(v[r][nt]));
      }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      // element offset within the tile's rows (past the range: dropped)
      const int is = (r0 + mt * 32 + g * 8 + r) * (int)N + cb;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const float x = v[r][nt] + bias[nt];
        const int o = is + nt * 32;
        if constexpr (MODE == EPI_BIAS_F32) {
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, x), out_f, o * 4, 0, 0);
        } else if constexpr (MODE == EPI_OPROJ) {
          const float y = res[slot][r][nt] + gate[nt] * x;
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, y), out_f, o * 4, 0, 0);
        } else if constexpr (MODE == EPI_UP) {
          const bf16 u = (bf16)gelu_tanh(x);
          __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, u), out_b, o * 2, 0, 0);
        } else if constexpr (MODE == EPI_DOWN) {
          const float y = res[slot][r][nt] + gate[nt] * x;
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, y), out_f, o * 4, 0, 0);
          const bf16 d = (bf16)(y - xin[slot][r][nt]);
          // out_t == null: a zero-length range drops the cached-residual store
          __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, d), out_b, o * 2, 0, 0);
          // column sums: rows past M count nowhere; the slot follows the camera boundary
          const int ro = roff + g * 8 + r;
          const float w = m0 + r0 + mt * 32 + g * 8 + r < M ? 1.f : 0.f;
          const float w1 = ro >= split[mt] ? w : 0.f, w0 = w - w1;
          if (g == 0 && r == 0) {
            sy[0][nt] = w0 * y;
            sy[1][nt] = w1 * y;
            sd[0][nt] = w0 * (float)d;
            sd[1][nt] = w1 * (float)d;
          } else {
            sy[0][nt] = fmaf(w0, y, sy[0][nt]);
            sy[1][nt] = fmaf(w1, y, sy[1][nt]);
            sd[0][nt] = fmaf(w0, (float)d, sd[0][nt]);
            sd[1][nt] = fmaf(w1, (float)d, sd[1][nt]);
          }
        }
      }
    }
    if constexpr (kXin) {
      if (g == 3) {
        // this 32-row block is complete: add the partner half-wave (the other
        // 16 rows), then half-wave hi writes slot hi
        const int hi = (r0 >> 2) & 1;
        const int rbo = ((rb0 + mt) * 2 + hi) * (int)N;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          float t[4] = {sy[0][nt], sy[1][nt], sd[0][nt], sd[1][nt]};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(t[k]), __float_as_uint(t[k]), false, false);
            t[k] = __uint_as_float(pr[0]) + __uint_as_float(pr[1]);
          }
          const int o = (rbo + cb + nt * 32) * 4;
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, hi ? t[1] : t[0]), part_y, o, 0, 0);
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, hi ? t[3] : t[2]), part_d, o, 0, 0);
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM.  Workgroup = 4 waves in a 2x2 arrangement; a wave owns an
// (MT*32) x (NT*32) sub-tile, i.e. MT x NT independent 32x32 accumulators of
// v_mfma_f32_32x32x16_bf16, so each 16-byte LDS fragment feeds several
// MFMAs.  K advances 32 per stage; the A and B stage tiles (64-byte rows) go
// from global memory straight into a 3-stage LDS ring (no staging
// registers, no LDS store instructions), two stages ahead of the MFMAs, and
// their 16-byte chunks are XOR-swizzled by (row / 4) so the rows a half-wave
// reads fall in distinct banks.  The 1-D grid is dealt to the XCDs in
// contiguous ranges of tiles, ordered in groups of 8 M-tiles x all N-tiles
// so concurrently resident tiles share A row blocks and B column blocks in
// the XCD's L2.
// ---------------------------------------------------------------------------
constexpr int kXcd = 8;
constexpr int GBK = 32;

template <int MT, int NT>
struct GemmTile {
  static constexpr int BM = 2 * MT * 32, BN = 2 * NT * 32;
  static constexpr int A_PER_T = BM * 4 / 256, B_PER_T = BN * 4 / 256;  // 16-byte chunks per thread and stage
  static constexpr int STAGE = (BM + BN) * GBK;                         // bf16 elements per stage
};

__device__ __forceinline__ int swz32(int row, int c) { return row * GBK + ((c ^ ((row >> 2) & 3)) << 3); }

// LDS bytes of the QKV epilogue: q / k stage the tile row-major [BM][BN + 8]
// bf16 followed by two [waves across N][BM] float arrays (partial sums of
// squares, scales); v transposes it through [BN][BM + 8] bf16.
template <int BM, int BN, int NT>
constexpr int qkv_epi_bytes() {
  return BM * (BN + 8) * 2 + 2 * (BN / (NT * 32)) * BM * 4 > BN * (BM + 8) * 2
             ? BM * (BN + 8) * 2 + 2 * (BN / (NT * 32)) * BM * 4
             : BN * (BM + 8) * 2;
}

// two floats as bf16 (round to nearest even), the first in the low half
__device__ __forceinline__ unsigned pack_bf16x2(float a, float b) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const f32x2 f = {a, b};
  return __builtin_bit_cast(unsigned, __builtin_convertvector(f, bf16x2));
}

template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// One halving step of a reduce-scatter across a lane bit: partner lanes (the
// DPP permutation CTRL pairs lanes that differ in that bit) swap halves of
// their HALF-pairs; the lane with the bit set keeps the upper half.
template <int CTRL, int HALF, int KP>
__device__ __forceinline__ void rs_step(float (&v)[KP], bool upper) {
#pragma unroll
  for (int i = 0; i < HALF; ++i) {
    const float send = upper ? v[i] : v[i + HALF], keep = upper ? v[i + HALF] : v[i];
    v[i] = keep + dpp_move<CTRL>(send);
  }
}

// Reduce-scatter of KP values per lane over the 32 lanes of each half-wave:
// afterwards lane lo (0..31) holds in v[j], j < KP / 32, the half-wave sum of
// value lo * KP / 32 + j.  Five halving steps, across lane bits 4 (the two
// 16-lane rows, permlane16 swap: row 0 keeps the lower half), 3 (row mirror),
// 2 (half-row mirror), 1 and 0 (quad permutations); 31 KP / 32 additions
// instead of the 5 KP of a butterfly per value.
template <int KP>
__device__ __forceinline__ void half_wave_reduce_scatter(float (&v)[KP], int lo) {
  static_assert(KP % 32 == 0, "whole values per lane");
#pragma unroll
  for (int i = 0; i < KP / 2; ++i) {
    const auto pr =
        __builtin_amdgcn_permlane16_swap(__float_as_uint(v[i]), __float_as_uint(v[i + KP / 2]), false, false);
    v[i] = __uint_as_float(pr[0]) + __uint_as_float(pr[1]);
  }
  rs_step<0x140, KP / 4>(v, (lo & 8) != 0);
  rs_step<0x141, KP / 8>(v, (lo & 4) != 0);
  rs_step<0x4E, KP / 16>(v, (lo & 2) != 0);
  rs_step<0xB1, KP / 32>(v, (lo & 1) != 0);
}

// QKV epilogue of a BM x BN tile (C = H*D columns per part, C % BN == 0, so a
// tile lies in one of q, k, v): bias; for q and k the per-(row, head) RMSNorm
// times the gain and the rotary embedding, stored bf16 to q_out / the key
// cache; for v the transpose through LDS into the V^T cache.  The tile's
// waves hold MT x NT accumulators each at rows wm*MT*32.., columns
// wn*NT*32..; NTHR threads; lds holds qkv_epi_bytes<BM, BN, NT>() bytes.
// accumulator element (mt, nt, g, r): tile row wm*MT*32 + mt*32 + g*8 + hi*4 + r,
// tile column wn*NT*32 + nt*32 + lo.  A wave's NT*32 = 64 columns lie in one
// head (D in {64, 128}).
template <int MT, int NT, int BM, int BN, int NTHR>
__device__ __forceinline__ void qkv_epilogue(const EpiArgs& e, const f32x16 (&acc)[MT][NT], char* lds, int m0, int n0,
                                             int M, int wm, int wn, int tid, int hi, int lo) {
  constexpr int WNW = BN / (NT * 32);  // waves across N
  static_assert(NT * 32 == 64, "one head per wave");
  const int C = e.H * e.D;
  const int lpart = n0 / C;            // a tile never straddles two column blocks
  const int part = lpart + e.part_base;  // 0 q, 1 k, 2 v
  const int head0 = (n0 - lpart * C) / e.D;
  // the accumulators plus bias as independent values (no 16-wide register
  // tuple stays live across the branches below)
  float x[MT][NT][16];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const float bv = e.bias[n0 + wn * NT * 32 + nt * 32 + lo];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        x[mt][nt][r] = acc[mt][nt][r] + bv;
        asm volatile("" : "+v"(x[mt][nt][r]));
      }
    }
  if (part < 2) {
    const float* gain = part == 0 ? e.gq : e.gk;
    const int hd = (wn * NT * 32) / e.D;  // the wave's head within the tile
    float gv[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) gv[nt] = gain[wn * NT * 32 + nt * 32 + lo - hd * e.D];
    // per (row, head) sum of squares over the head's D columns: the lane's
    // NT columns, then the half-wave's 32 lanes (value k = (mt*4 + g)*4 + r is
    // row wm*MT*32 + mt*32 + g*8 + hi*4 + r), then the D / 64 waves of the head
    constexpr int KV = MT * 16, KP = (KV + 31) / 32 * 32, KL = KP / 32;
    float p[KP];
#pragma unroll
    for (int k = 0; k < KP; ++k) {
      float q = 0.f;
      if (k < KV) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) q += x[k >> 4][nt][k & 15] * x[k >> 4][nt][k & 15];
      }
      p[k] = q;
    }
    half_wave_reduce_scatter(p, lo);
    float* red = reinterpret_cast<float*>(lds + BM * (BN + 8) * 2);  // [WNW][BM] the waves' partial sums
    float* scl = red + WNW * BM;                 // [WNW][BM] the scales each wave reads
    const int rw = wm * MT * 32 + hi * 4;        // the half-wave's first row
#pragma unroll
    for (int j = 0; j < KL; ++j) {
      const int k = lo * KL + j;
      if (k < KV) red[wn * BM + rw + (k >> 4) * 32 + ((k >> 2) & 3) * 8 + (k & 3)] = p[j];
    }
    __syncthreads();
    const int wph = e.D / (NT * 32), w0 = wn / wph * wph;  // the head's waves
#pragma unroll
    for (int j = 0; j < KL; ++j) {
      const int k = lo * KL + j;
      if (k < KV) {
        const int row = rw + (k >> 4) * 32 + ((k >> 2) & 3) * 8 + (k & 3);
        float sum = 0.f;
        for (int w = w0; w < w0 + wph; ++w) sum += red[w * BM + row];
        scl[wn * BM + row] = 1.0f / sqrtf(sum / (float)e.D + 1e-6f);
      }
    }
    __syncthreads();
    // rotary embedding, per column of this lane: the table entry of its pair
    // at axis position 0, the entry stride per position, the position's bit
    // offset in the packed row coordinates
    const bool rope = e.rope.tab != nullptr;
    int rbase[NT], rstride[NT], rshift[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      int pair = (wn * NT * 32 + nt * 32 + lo - hd * e.D) >> 1, a = 0;
      if (rope && pair >= e.rope.np[0]) {
        pair -= e.rope.np[0];
        a = 1;
        if (pair >= e.rope.np[1]) {
          pair -= e.rope.np[1];
          a = 2;
        }
      }
      rbase[nt] = rope ? e.rope.off[a] + pair : 0;
      rstride[nt] = rope ? e.rope.np[a] : 0;
      rshift[nt] = 10 * a;
    }
    // Normalise (and rotate) one group of 4 rows at a time and put it in
    // LDS as bf16, row-major (the sums and scales sit behind the tile); the
    // tile then leaves in 16-byte row chunks: tile row t of head h to
    // q_out[h][m0 + t] or to token kv_off + m0 + t of the key cache.  The
    // LDS offsets of a lane's values are compile-time immediates.
    const float* sl4 = scl + wn * BM + rw;  // scales of the half-wave's rows
    bf16* stg = reinterpret_cast<bf16*>(lds);
    constexpr int SW = BN + 8;
    bf16* sl = stg + rw * SW + wn * NT * 32 + lo;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        // scales of rows g*8 + hi*4 + 0..3 of 32-row block mt: one 16-byte read
        const f32x4 sc = *reinterpret_cast<const f32x4*>(sl4 + mt * 32 + g * 8);
        float y[4][NT];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) y[r][nt] = x[mt][nt][g * 4 + r] * sc[r] * gv[nt];
        if (rope) {
          // the group's table entries are loaded together (one wait, not one per value)
          int packed[4];
#pragma unroll
          for (int r = 0; r < 4; ++r)  // rows past M: clamped, never stored
            packed[r] = e.rope.pos[min(m0 + rw + mt * 32 + g * 8 + r, M - 1)];
          float2 cs[4][NT];
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
              cs[r][nt] = e.rope.tab[rbase[nt] + ((packed[r] >> rshift[nt]) & 1023) * rstride[nt]];
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              // rotary pair (dd & ~1, dd | 1) = lanes (lo & ~1, lo | 1) of the same row, swapped
              // by a DPP quad permutation [1, 0, 3, 2]: (a, b) -> (a c - b s, a s + b c)
              const float pv = dpp_move<0xB1>(y[r][nt]);
              y[r][nt] = y[r][nt] * cs[r][nt].x + ((lo & 1) ? pv : -pv) * cs[r][nt].y;
            }
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int r = 0; r < 4; r += 2) {
            const unsigned w = pack_bf16x2(y[r][nt], y[r + 1][nt]);
            sl[(mt * 32 + g * 8 + r) * SW + nt * 32] = __builtin_bit_cast(bf16, (unsigned short)w);
            sl[(mt * 32 + g * 8 + r + 1) * SW + nt * 32] = __builtin_bit_cast(bf16, (unsigned short)(w >> 16));
          }
      }
    __syncthreads();
    constexpr int CPR = BN / 8, RPI = NTHR / CPR, ITER = BM / RPI;
    static_assert(NTHR % CPR == 0 && BM % RPI == 0, "whole rows per pass");
    const int cc = tid % CPR, row0 = tid / CPR;
    const int hc = cc * 8 / e.D, dd = cc * 8 - hc * e.D;
    const long long hh = head0 + hc;
    const int rows = min(BM, M - m0);
    bf16* dst = part == 0 ? reinterpret_cast<bf16*>(e.q_out) + (hh * e.Mpad + m0 + row0) * e.D + dd
                          : reinterpret_cast<bf16*>(e.k_cache) + (hh * e.Lcap + e.kv_off + m0 + row0) * e.D + dd;
    u32x4 ch[ITER];
#pragma unroll
    for (int it = 0; it < ITER; ++it) ch[it] = *reinterpret_cast<const u32x4*>(stg + (row0 + it * RPI) * SW + cc * 8);
#pragma unroll
    for (int it = 0; it < ITER; ++it)
      if (row0 + it * RPI < rows) *reinterpret_cast<u32x4*>(dst + (long long)it * RPI * e.D) = ch[it];
  } else {
    // V^T: row head0*D + c of the cache holds column c of the tile, tokens
    // contiguous.  The tile goes through LDS column-major, each column's
    // token t at position s + t with s = (kv_off + m0) mod 8, so that 8-token
    // chunks of a column (16 bytes at positions 8q..8q+7) start at a token
    // index that is a multiple of 8 in the cache: 16-byte aligned stores.
    // A lane holds tokens g*8 + hi*4 + 0..3 of its column: one 8-byte LDS
    // write when s is a multiple of 4.
    bf16* vt = reinterpret_cast<bf16*>(lds);  // [BN][VS]
    constexpr int VS = BM + 8;
    const int t0 = e.kv_off + m0;  // the tile's first token in the cache
    const int s = t0 & 7;
    bf16* vl = vt + (wn * NT * 32 + lo) * VS + s + wm * MT * 32 + hi * 4;
    if ((s & 3) == 0) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int g = 0; g < 4; ++g)
            *reinterpret_cast<uint2*>(vl + nt * 32 * VS + mt * 32 + g * 8) =
                make_uint2(pack_bf16x2(x[mt][nt][g * 4], x[mt][nt][g * 4 + 1]),
                           pack_bf16x2(x[mt][nt][g * 4 + 2], x[mt][nt][g * 4 + 3]));
    } else {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int r = 0; r < 4; ++r) vl[nt * 32 * VS + mt * 32 + g * 8 + r] = (bf16)x[mt][nt][g * 4 + r];
    }
    __syncthreads();
    // chunk q of column c: tile rows 8q - s .. 8q - s + 7, cache tokens
    // t0 - s + 8q ..; rows outside [0, rows) are not stored
    constexpr int QC = BM / 8 + 1, VIT = (BN * QC + NTHR - 1) / NTHR;
    const int rows = min(BM, M - m0);
    bf16* vbase = reinterpret_cast<bf16*>(e.vt_cache) + (long long)head0 * e.D * e.Lcap + (t0 - s);
    const bool vec = ((reinterpret_cast<unsigned long long>(e.vt_cache) | ((unsigned long long)e.Lcap * 2)) & 15) == 0;
    u32x4 ch[VIT];
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int idx = tid + it * NTHR;
      if (idx < BN * QC) {
        const int c = idx / QC, q = idx - c * QC;
        ch[it] = *reinterpret_cast<const u32x4*>(vt + c * VS + 8 * q);
      }
    }
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int idx = tid + it * NTHR;
      if (idx < BN * QC) {
        const int c = idx / QC, q = idx - c * QC;
        const int r0 = 8 * q - s;
        bf16* dst = vbase + (long long)c * e.Lcap + 8 * q;
        if (vec && r0 >= 0 && r0 + 8 <= rows) {
          *reinterpret_cast<u32x4*>(dst) = ch[it];
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (r0 + i >= 0 && r0 + i < rows)
              dst[i] = __builtin_bit_cast(bf16, (unsigned short)(ch[it][i >> 1] >> (16 * (i & 1))));
        }
      }
    }
  }
}

template <int MODE, int MT, int NT>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(const bf16* __restrict__ A, const bf16* __restrict__ W,
                                                           int M, int N, int K, EpiArgs e,
                                                           const int* __restrict__ flag) {
  if (flag != nullptr && *flag) return;
  typedef GemmTile<MT, NT> T;
  constexpr int MAIN_BYTES = 3 * T::STAGE * 2;
  constexpr int EPI_BYTES = MODE == EPI_QKV ? qkv_epi_bytes<T::BM, T::BN, NT>() : 0;
  constexpr int LDS_BYTES = MAIN_BYTES > EPI_BYTES ? MAIN_BYTES : EPI_BYTES;
  __shared__ __attribute__((aligned(16))) char lds[LDS_BYTES];
  bf16* sbuf = reinterpret_cast<bf16*>(lds);

  const int n_tm = (M + T::BM - 1) / T::BM, n_tn = N / T::BN;
  const int total = n_tm * n_tn;
  const int per_xcd = (total + kXcd - 1) / kXcd;
  const int t = (blockIdx.x % kXcd) * per_xcd + blockIdx.x / kXcd;
  if (t >= total) return;
  constexpr int GM = 8;
  const int in_group = GM * n_tn;
  const int first_m = (t / in_group) * GM;
  const int gm = min(GM, n_tm - first_m);
  const int tm = first_m + (t % in_group) % gm, tn = (t % in_group) / gm;
  const int m0 = tm * T::BM, n0 = tn * T::BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int hi = lane >> 5, lo = lane & 31;
  const bf16* Ab = A + (long long)m0 * K;
  const bf16* Wb = W + (long long)n0 * K;
  f32x16 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int KT = K / GBK;
  // Stages go global -> LDS directly (global_load_lds_dwordx4): one wave
  // instruction fills 1 KB of LDS lane-linearly, i.e. 16 rows x 4 chunks; a
  // lane fetches the logical chunk that the swizzle places at its position.
  constexpr int A_INSTR = T::BM / 16 / 4, B_INSTR = T::BN / 16 / 4;  // per wave
  constexpr int LOADS = A_INSTR + B_INSTR;
  const int lrow = lane >> 2, lpc = lane & 3;
  auto issue = [&](int kt, int buf) __attribute__((always_inline)) {
    bf16* sa = sbuf + buf * T::STAGE;
    bf16* sb = sa + T::BM * GBK;
#pragma unroll
    for (int i = 0; i < A_INSTR; ++i) {
      const int I = wave + 4 * i, row = I * 16 + lrow, c = lpc ^ ((row >> 2) & 3);
      __builtin_amdgcn_global_load_lds(Ab + (long long)row * K + kt * GBK + c * 8, sa + I * 512, 16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < B_INSTR; ++i) {
      const int I = wave + 4 * i, row = I * 16 + lrow, c = lpc ^ ((row >> 2) & 3);
      __builtin_amdgcn_global_load_lds(Wb + (long long)row * K + kt * GBK + c * 8, sb + I * 512, 16, 0, 0);
    }
  };
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const bf16* sa = sbuf + buf * T::STAGE;
    const bf16* sb = sa + T::BM * GBK;
#pragma unroll
    for (int kk = 0; kk < GBK / 16; ++kk) {
      const int c = kk * 2 + hi;
      bf16x8 a[MT], b[NT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) a[mt] = *reinterpret_cast<const bf16x8*>(&sa[swz32(wm * MT * 32 + mt * 32 + lo, c)]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) b[nt] = *reinterpret_cast<const bf16x8*>(&sb[swz32(wn * NT * 32 + nt * 32 + lo, c)]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mt], b[nt], acc[mt][nt], 0, 0, 0);
    }
  };
  // vmcnt(n) with the other counters left at their maximum (gfx9 encoding)
#define XC_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((0x3f70) | ((n) & 15) | (((n) >> 4) << 14))

  // Stage k lives in LDS buffer k mod 3; stage k+2 is requested while stage k
  // is multiplied, and stage k+1 (requested one step earlier) is waited for
  // before the barrier.  Requests past the last stage repeat it (in bounds,
  // into a buffer nobody reads again), so every step is the same code.
  issue(0, 0);
  issue(min(1, KT - 1), 1);
  XC_WAIT_VMCNT(LOADS);
  __syncthreads();
  auto step = [&](int kt, int b0, int b2) __attribute__((always_inline)) {  // b0 = kt mod 3, b2 = (kt+2) mod 3
    issue(min(kt + 2, KT - 1), b2);
    compute(b0);
    XC_WAIT_VMCNT(LOADS);
    __syncthreads();
  };
  int kt = 0;
  for (; kt + 2 < KT; kt += 3) {
    step(kt, 0, 2);
    step(kt + 1, 1, 0);
    step(kt + 2, 2, 1);
  }
  if (kt < KT) step(kt, 0, 2);
  if (kt + 1 < KT) step(kt + 1, 1, 0);
  XC_WAIT_VMCNT(0);  // the epilogue may reuse the LDS: no request may still be landing
  __syncthreads();
#undef XC_WAIT_VMCNT

  // accumulator element (mt, nt, g, r): tile row wm*MT*32 + mt*32 + g*8 + hi*4 + r,
  // tile column wn*NT*32 + nt*32 + lo
  if constexpr (MODE == EPI_QKV) {
    qkv_epilogue<MT, NT, T::BM, T::BN, 256>(e, acc, lds, m0, n0, M, wm, wn, tid, hi, lo);
  } else {
    tile_epilogue<MODE, MT, NT>(e, acc, m0, wm * MT * 32 + hi * 4, n0 + wn * NT * 32 + lo, M, T::BM);
  }
}

// ---------------------------------------------------------------------------
// Wide bf16 MFMA GEMM: one workgroup of 8 waves per CU owns a 256 x BN tile,
// its waves in a WMW x (8 / WMW) arrangement: 256 x 256 tiles as 2 x 4 waves
// of 128 x 64 (4 x 2 accumulators each, as in gemm_bf16_kernel), 256 x 192
// tiles as 4 x 2 waves of 64 x 96 (2 x 3).  Stages are 64 deep: every DMA
// request fetches 128 contiguous bytes of a row (a whole cache line; the
// request stream measures 14.6 TB/s with the 64-byte segments of 32-deep
// stages against 24.5 TB/s with 128-byte ones, xc_lds_dma_rate), and per
// output element a 256 x 256 tile moves a third fewer operand bytes than two
// 256 x 128 tiles.  The weights have a ring of three stage slots and the
// activations one of two (160 KB for 256 x 256 tiles, 136 KB for 256 x 192):
// weights are requested two steps ahead, activations one step ahead, both at
// the top of a step while the current stage is multiplied.  LDS rows are 128
// bytes with their 16-byte chunks XOR-swizzled (swz8) so the 32 rows a
// half-wave reads at one chunk position fall in distinct banks.  256 x 256
// tiles serve the QKV and MLP-up projections (N % 256 == 0, K % 64 == 0, and
// C % 256 == 0 for QKV), 256 x 192 tiles the output and MLP-down projections
// (N % 192 == 0).
// ---------------------------------------------------------------------------
constexpr int WBM = 256, WBK = 64;

// physical 16-byte chunk of logical chunk c in a 128-byte LDS row r (an
// involution in c): any 8 consecutive rows at distinct chunks, any 16 at
// distinct (row parity, chunk) pairs
__device__ __forceinline__ int swz8(int r, int c) { return c ^ ((r & 7) ^ ((r >> 3) & 1)); }

// one 16-byte chunk per lane, global -> LDS; lane l lands at byte 16 l of the
// wave's 1 KB block
__device__ __forceinline__ void dma16(const bf16* src, bf16* lds_block) {
  __builtin_amdgcn_global_load_lds(src, lds_block, 16, 0, 0);
}

template <int MODE, int BN, int WMW>
__global__ __launch_bounds__(512, 1) void gemm_bf16_wide(const bf16* __restrict__ A, const bf16* __restrict__ W,
                                                         int M, int N, int K, EpiArgs e,
                                                         const int* __restrict__ flag) {
  if (flag != nullptr && *flag) return;
  constexpr int WNW = 8 / WMW, MT = WBM / 32 / WMW, NT = BN / 32 / WNW;
  static_assert(MT * 32 * WMW == WBM && NT * 32 * WNW == BN && BN % 64 == 0, "wide tile shape");
  constexpr int ASLOT = WBM * WBK, WSLOT = BN * WBK;  // bf16 elements of one A / W stage slot
  constexpr int MAIN_BYTES = (2 * ASLOT + 3 * WSLOT) * 2;  // A ring of 2, W ring of 3
  constexpr int EPI_BYTES = MODE == EPI_QKV ? qkv_epi_bytes<WBM, BN, NT>() : 0;
  constexpr int LDS_BYTES = MAIN_BYTES > EPI_BYTES ? MAIN_BYTES : EPI_BYTES;
  __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES];
  bf16* sbuf = reinterpret_cast<bf16*>(lds);

  const int n_tm = (M + WBM - 1) / WBM, n_tn = N / BN;
  const int total = n_tm * n_tn;
  const int per_xcd = (total + kXcd - 1) / kXcd;
  const int t = (blockIdx.x % kXcd) * per_xcd + blockIdx.x / kXcd;
  if (t >= total) return;
  constexpr int GM = 8;
  const int in_group = GM * n_tn;
  const int first_m = (t / in_group) * GM;
  const int gm = min(GM, n_tm - first_m);
  const int tm = first_m + (t % in_group) % gm, tn = (t % in_group) / gm;
  const int m0 = tm * WBM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WNW, wn = wave % WNW;
  const int hi = lane >> 5, lo = lane & 31;
  const bf16* Ab = A + (long long)m0 * K;
  const bf16* Wb = W + (long long)n0 * K;
  // DMA request I of an operand (A: 0..31, W: 0..BN/8-1) fills its rows
  // 8I .. 8I+7 lane-linearly (lane l: row 8I + l/8, physical chunk l%8, which
  // holds the logical chunk swz8(row, l%8)); wave w issues I = w + 8i
  int goff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = (wave + 8 * i) * 8 + (lane >> 3);
    goff[i] = row * K + swz8(row, lane & 7) * 8;
  }
  // fragment reads: row lo (plus multiples of 32), logical chunk 2 kk + hi;
  // the swizzle depends on the row's low 4 bits only
  int foff[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) foff[kk] = lo * WBK + swz8(lo, 2 * kk + hi) * 8;
  f32x16 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int KT = K / WBK;
  auto issue_a = [&](int kt, int slot) __attribute__((always_inline)) {
    bf16* sa = sbuf + slot * ASLOT;
#pragma unroll
    for (int i = 0; i < WBM / 64; ++i) dma16(Ab + goff[i] + kt * WBK, sa + (wave + 8 * i) * 512);
  };
  auto issue_w = [&](int kt, int slot) __attribute__((always_inline)) {
    bf16* sb = sbuf + 2 * ASLOT + slot * WSLOT;
#pragma unroll
    for (int i = 0; i < BN / 64; ++i) dma16(Wb + goff[i] + kt * WBK, sb + (wave + 8 * i) * 512);
  };
  auto compute = [&](int aslot, int wslot) __attribute__((always_inline)) {
    const bf16* sa = sbuf + aslot * ASLOT + (wm * MT * 32) * WBK;
    const bf16* sb = sbuf + 2 * ASLOT + wslot * WSLOT + (wn * NT * 32) * WBK;
#pragma unroll
    for (int kk = 0; kk < WBK / 16; ++kk) {
      bf16x8 a[MT], b[NT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) a[mt] = *reinterpret_cast<const bf16x8*>(sa + mt * 32 * WBK + foff[kk]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) b[nt] = *reinterpret_cast<const bf16x8*>(sb + nt * 32 * WBK + foff[kk]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mt], b[nt], acc[mt][nt], 0, 0, 0);
    }
  };
  // A(k) lives in A slot k mod 2, W(k) in W slot k mod 3: the weights, which
  // stream from HBM (the activations were just written and sit in the
  // caches), are requested two steps ahead.  Step k requests A(k+1) and then
  // W(k+2) (their slots were released by the barrier that ended step k-1),
  // multiplies stage k, and waits for everything but the W(k+2) requests
  // (vmcnt counts in issue order).  The barrier's workgroup release fence
  // then also waits for those on this chip; a barrier without the fence,
  // which leaves them in flight, measured the same (they land within a
  // step), so the plain __syncthreads stays.
#define XC_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((0x3f70) | ((n) & 15) | (((n) >> 4) << 14))
  constexpr int WREQ = BN / 64;
  issue_w(0, 0);
  issue_a(0, 0);
  if (KT > 1) {
    issue_w(1, 1);
    XC_WAIT_VMCNT(WREQ);
  } else {
    XC_WAIT_VMCNT(0);
  }
  __syncthreads();
  auto step = [&](int kt, int as, int ws) __attribute__((always_inline)) {
    if (kt + 1 < KT) issue_a(kt + 1, as ^ 1);
    if (kt + 2 < KT) issue_w(kt + 2, ws == 0 ? 2 : ws - 1);
    compute(as, ws);
    if (kt + 2 < KT) XC_WAIT_VMCNT(WREQ); else XC_WAIT_VMCNT(0);
    __syncthreads();
  };
  int kt = 0;
  for (; kt + 5 < KT; kt += 6) {
    step(kt, 0, 0);
    step(kt + 1, 1, 1);
    step(kt + 2, 0, 2);
    step(kt + 3, 1, 0);
    step(kt + 4, 0, 1);
    step(kt + 5, 1, 2);
  }
  for (; kt < KT; ++kt) step(kt, kt & 1, kt % 3);
#undef XC_WAIT_VMCNT

  if constexpr (MODE == EPI_QKV) {
    qkv_epilogue<MT, NT, WBM, BN, 512>(e, acc, lds, m0, n0, M, wm, wn, tid, hi, lo);
  } else {
    tile_epilogue<MODE, MT, NT>(e, acc, m0, wm * MT * 32 + hi * 4, n0 + wn * NT * 32 + lo, M, WBM);
  }
}

template <int MODE>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, const float* __restrict__ W,
                                                       int M, int N, int K, EpiArgs e, const int* __restrict__ flag) {
  if (flag != nullptr && *flag) return;
  __shared__ float sA[16][68];
  __shared__ float sW[16][68];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = threadIdx.x + 256 * i, r = idx >> 4, k = idx & 15;
      sA[k][r] = (m0 + r < M && k0 + k < K) ? A[(long long)(m0 + r) * K + k0 + k] : 0.f;
      sW[k][r] = (n0 + r < N && k0 + k < K) ? W[(long long)(n0 + r) * K + k0 + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = sA[k][ty * 4 + i];
        b[i] = sW[k][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
      if (row < M && col < N) epilogue<MODE, float>(e, row, col, acc[i][j]);
    }
}

int cu_count() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus = n;
  }
  return cus;
}

// Rows per M-tile for an M x N product: the tile height (64*MT) whose tile
// count best fills whole rounds of resident workgroups (2 per CU); 64-row
// tiles only where even 128-row tiles leave CUs without one (small
// products, e.g. 768 tokens), since they move more operand bytes per flop.
int pick_mt(int M, int N) {
  const int slots = 2 * cu_count();
  int best = 4;
  double best_cost = 1e300;
  for (int mt = 4; mt >= 2; --mt) {
    const long long tiles = (long long)((M + 64 * mt - 1) / (64 * mt)) * (N / 128);
    const long long rounds = (tiles + slots - 1) / slots;
    const double cost = (double)rounds * mt;  // one round costs in proportion to the tile height
    if (cost < best_cost - 1e-9) {
      best_cost = cost;
      best = mt;
    }
  }
  if (best == 2 && (long long)((M + 127) / 128) * (N / 128) < cu_count()) best = 1;
  return best;
}

template <int MODE, int MT>
void launch_bf16(const void* A, const void* W, int M, int N, int K, const EpiArgs& e, const int* flag, hipStream_t st) {
  typedef GemmTile<MT, 2> T;
  const int tiles = ((M + T::BM - 1) / T::BM) * (N / T::BN);
  const int grid = (tiles + kXcd - 1) / kXcd * kXcd;
  gemm_bf16_kernel<MODE, MT, 2><<<grid, 256, 0, st>>>((const bf16*)A, (const bf16*)W, M, N, K, e, flag);
}

// Whether wide 256 x BN tiles beat the two-workgroup kernel for an M x N
// product: a round's time taken in proportion to the tile area a CU works
// through (two resident (64*MT) x 128 tiles share a CU), the wide kernel
// 12% more efficient per flop (the multi-camera QKV product: 122.8 against
// 137.5 us in one round-count class).  Small token counts leave most CUs
// idle under wide tiles (768 tokens: 18 tiles of 256 x 256 for the QKV
// product), where the smaller tiles win.
bool wide_pays(int M, int N, int BN) {
  const long long cus = cu_count();
  const long long wt = (long long)((M + WBM - 1) / WBM) * (N / BN);
  const double wide = (double)((wt + cus - 1) / cus) * WBM * BN / 1.12;
  const int mt = pick_mt(M, N);
  const long long t2 = (long long)((M + 64 * mt - 1) / (64 * mt)) * (N / 128);
  const double two = (double)((t2 + 2 * cus - 1) / (2 * cus)) * (64.0 * mt * 128.0) * 2.0;
  return wide <= two;
}

template <int MODE, int BN, int WMW>
void launch_wide(const void* A, const void* W, int M, int N, int K, const EpiArgs& e, const int* flag,
                 hipStream_t st) {
  const int tiles = ((M + WBM - 1) / WBM) * (N / BN);
  const int grid = (tiles + kXcd - 1) / kXcd * kXcd;
  gemm_bf16_wide<MODE, BN, WMW><<<grid, 512, 0, st>>>((const bf16*)A, (const bf16*)W, M, N, K, e, flag);
}

template <int MODE>
void launch_mode(int dtype, const void* A, const void* W, int M, int N, int K, const EpiArgs& e, const int* flag,
                 hipStream_t st) {
  if (dtype == 1) {
    // Wide tiles, measured at the multi-camera shapes: the QKV and MLP-up
    // products on 256 x 256 (QKV 115 vs 140 us, MLP-up 156 vs 190 us against
    // the two-workgroup kernel); the output and MLP-down projections on
    // 256 x 192 (the same box in one call: 49.6 vs 51.3 us and 145.6 vs
    // 147.6 us in the full pass against a persistent 4-wave kernel with
    // 32-deep stages, which this replaced, and 49.8 vs 54.7 us and 146.1 vs
    // 163.2 us against the two-workgroup kernel on 192 x 128 tiles; 256 x 256
    // tiles leave 168 tiles for 256 CUs at hidden 1536).  Other widths: the
    // two-workgroup kernel (at hidden 2048 it measured 445 vs 451 us for MLP
    // down and 132 vs 136 us for the output projection against 256 x 256
    // wide tiles), and products whose wide tiles leave the chip underfilled
    // (wide_pays).
    if constexpr (MODE == EPI_QKV || MODE == EPI_UP) {
      if (N % 256 == 0 && K % WBK == 0 && (MODE != EPI_QKV || (e.H * e.D) % 256 == 0) && wide_pays(M, N, 256)) {
        launch_wide<MODE, 256, 2>(A, W, M, N, K, e, flag, st);
        return;
      }
    } else {
      if (N % 192 == 0 && K % WBK == 0 && wide_pays(M, N, 192)) {
        launch_wide<MODE, 192, 4>(A, W, M, N, K, e, flag, st);
        return;
      }
    }
    switch (pick_mt(M, N)) {
      case 4: launch_bf16<MODE, 4>(A, W, M, N, K, e, flag, st); break;
      case 3: launch_bf16<MODE, 3>(A, W, M, N, K, e, flag, st); break;
      case 2: launch_bf16<MODE, 2>(A, W, M, N, K, e, flag, st); break;
      default: launch_bf16<MODE, 1>(A, W, M, N, K, e, flag, st); break;
    }
  } else {
    dim3 grid((N + 63) / 64, (M + 63) / 64);
    gemm_f32_kernel<MODE><<<grid, 256, 0, st>>>((const float*)A, (const float*)W, M, N, K, e, flag);
  }
}

}  // namespace

// bf16 requirements (checked by the caller): N % 128 == 0, K % 32 == 0, A has
// at least roundup(M, 256) rows allocated; EPI_QKV needs C % 128 == 0 and
// D in {64, 128}.
void launch_gemm(int dtype, EpiMode mode, const void* A, const void* W, int M, int N, int K, const EpiArgs& e,
                 const int* flag, hipStream_t st) {
  switch (mode) {
    case EPI_BIAS_F32: launch_mode<EPI_BIAS_F32>(dtype, A, W, M, N, K, e, flag, st); break;
    case EPI_OPROJ: launch_mode<EPI_OPROJ>(dtype, A, W, M, N, K, e, flag, st); break;
    case EPI_UP: launch_mode<EPI_UP>(dtype, A, W, M, N, K, e, flag, st); break;
    case EPI_DOWN: launch_mode<EPI_DOWN>(dtype, A, W, M, N, K, e, flag, st); break;
    case EPI_QKV: launch_mode<EPI_QKV>(dtype, A, W, M, N, K, e, flag, st); break;
  }
}

}  // namespace xc
