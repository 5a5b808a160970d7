// Self-attention of the chunk's queries over the rolling key/value window
// (current chunk plus the kept past chunks), softmax(q k^T / sqrt(d)) v per
// head, no mask.  Keys of all visible chunks are contiguous rows [0, Lk) of
// the per-head cache, so the kernel sees one key range.
//
// bf16 path (flash-style, one pass over the keys with an online softmax):
//   * workgroup = 8 waves = 256 queries of one head (one workgroup per CU,
//     two waves per SIMD); each wave owns 32 queries whose Q fragments stay in
//     registers for the whole key loop, and the 8 waves share every staged
//     K / V^T tile;
//   * per 64-key tile, S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (keys on the
//     MFMA rows, queries on the columns), so each lane holds 32 scores of ONE
//     query: the running max/sum and the output rescale are lane-local except
//     one exchange with the partner lane (lane ^ 32);
//   * O^T += V^T P^T on the same MFMA: the V cache is stored transposed
//     ([d][keys]) so a lane's 8-key operand is one 16-byte LDS read, and the K
//     tile rows are permuted in LDS so that the score registers of each lane
//     are exactly the 8 consecutive keys the P operand needs (no shuffles);
//   * K and V^T tiles are double-buffered in LDS, filled by LDS-DMA;
//     scores are scaled into the log2 domain by one FMA and exponentiated
//     with exp2; the softmax denominator sums the bf16 probabilities that the
//     P.V product consumes (two per dot2 instruction); accumulation is float.
// fp32 path: one wave per (query, head), plain online softmax.
#include "xc_internal.h"

#include <math.h>

namespace xc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

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

// vmcnt(0), the other counters left alone (gfx9 encoding)
#define XC_WAIT_VMCNT0() __builtin_amdgcn_s_waitcnt(0x3f70)
// one 16-byte chunk per lane, global -> LDS (lane l lands at byte 16 l of
// the wave's 1 KB block)
__device__ __forceinline__ void dma16(const char* src, bf16* lds_block) {
  __builtin_amdgcn_global_load_lds(src, lds_block, 16, 0, 0);
}

constexpr int kXcds = 8;
constexpr int kWaves = 8;            // waves per attention workgroup
constexpr int kQT = 32 * kWaves;     // queries per attention workgroup

// Workspace floats of one (item, key split) piece: the piece's output
// normalised by its own softmax sum, bf16 [kQT][D], then its running max and
// sum, float [kQT] each.
__host__ __device__ constexpr long long piece_floats(int D) { return (long long)kQT * D / 2 + 2 * kQT; }

__device__ __forceinline__ float partner_max(float x) {
  // max(x, x of lane ^ 32): v_permlane32_swap exchanges the two half-waves
  // (a VALU operation, no LDS round trip)
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float partner_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Work distribution.  An item is (head, 256-query tile); its key tiles are
// split into S equal chunks, S chosen by the launcher so that the units
// (item, chunk) fill whole rounds of resident workgroups (one per CU).  Units
// are ordered [head][chunk][query tile] and dealt to the 8 XCDs (each with
// its own L2) in contiguous ranges (workgroups are dispatched round-robin
// over the XCDs, so workgroup b takes unit (b mod 8) * per_xcd + b / 8): the
// workgroups resident on one XCD then stream the same key/value chunk of one
// head at about the same time.  With S = 1 a unit writes the normalised
// output; otherwise it leaves (O unnormalised, running max, running sum) in
// the workspace and the merge kernel combines the S pieces of each item.
//
// Software pipeline, per wave and key tile j:
//   S(j+1) = K(j+1) Q^T on the MFMA pipe, while the VALU runs the softmax of
//   S(j); then O^T += V(j)^T P(j)^T.  K runs one tile ahead of V in LDS:
//   iteration j reads K(j+1) and V(j) and refills K(j+2) and V(j+1).
template <int D>
__global__ __launch_bounds__(64 * kWaves, 1) void attn_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ Kc,
                                                           const bf16* __restrict__ Vt, bf16* __restrict__ O, int L,
                                                           int Mpad, int Lcap, int Lk, int H, int n_qt, int n_split,
                                                           float sl2, float* __restrict__ ws,
                                                           const int* __restrict__ flag) {
  if (flag != nullptr && *flag) return;
  constexpr int KCH = D / 8;                // 16-byte chunks per key row
  constexpr int KCG = KCH / 8;              // groups of 8 chunks per K row
  constexpr int KB = 8 * KCG / kWaves;      // K DMA blocks per wave and tile
  constexpr int VB = D / 8 / kWaves;        // V^T DMA blocks per wave and tile
  static_assert(KB >= 1 && VB >= 1, "staging layout");
  constexpr int DT = D / 32;                // 32-row output tiles (head dims)
  // K and V^T tiles go global -> LDS by DMA (no register staging), in 1 KB
  // blocks of 8 rows x 8 sixteen-byte chunks: row r, chunk c sits in block
  // (r / 8, c / 8) at slot ((c % 8) ^ (r / 8 % 2)) * 8 + r % 8.  A DMA
  // instruction fills one block (each lane fetches the chunk its slot holds:
  // 128-byte row segments), the 16 rows a quarter-wave reads at one chunk
  // fall in 16 distinct 16-byte bank groups without padding, and every
  // fragment address is a per-lane base plus a compile-time offset.
  // Four separate arrays: the compiler then tells a DMA into one buffer from
  // fragment reads of the other and does not wait for the DMA before them
  __shared__ __attribute__((aligned(1024))) bf16 sK0[64 * D];
  __shared__ __attribute__((aligned(1024))) bf16 sK1[64 * D];
  __shared__ __attribute__((aligned(1024))) bf16 sV0[D * 64];
  __shared__ __attribute__((aligned(1024))) bf16 sV1[D * 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hi = lane >> 5, lo = lane & 31;
  const int C = H * D;
  const int NT = (Lk + 63) / 64;
  const int units = H * n_split * n_qt;
  const int per_xcd = (units + kXcds - 1) / kXcds;
  const int unit = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (unit >= units) return;
  const int h = unit / (n_split * n_qt);
  const int rem = unit - h * n_split * n_qt;
  const int kc = rem / n_qt, qt = rem - kc * n_qt;
  const int k0 = (int)((long long)kc * NT / n_split), k1 = (int)((long long)(kc + 1) * NT / n_split);
  const int q0 = qt * kQT + wave * 32;
  // Waves whose 32 queries all lie past L (in a ragged last query tile) have
  // nothing to compute: they only stage their share of the K / V^T tiles, in
  // a loop of their own with the same barriers (a branch inside the shared
  // loop instead costs the other waves registers).
  const bool live = __builtin_amdgcn_readfirstlane(q0) < L;

  // source byte offsets (within a tile) of the blocks this wave fills: lane l
  // lands at slot l, i.e. row 8 rg + l % 8 and chunk 8 cg + ((l / 8) ^ (rg & 1));
  // LDS row R of a K tile holds key key_of_row(R / 32, R % 32)
  int kg[KB], vg[VB];
#pragma unroll
  for (int i = 0; i < KB; ++i) {
    const int B = wave + kWaves * i, rg = B / KCG, cg = B % KCG;
    const int R = rg * 8 + (lane & 7), c = cg * 8 + ((lane >> 3) ^ (rg & 1));
    kg[i] = (key_of_row(R >> 5, R & 31) * D + c * 8) * 2;
  }
#pragma unroll
  for (int i = 0; i < VB; ++i) {
    const int rg = wave + kWaves * i;
    const int d = rg * 8 + (lane & 7), c = (lane >> 3) ^ (rg & 1);
    vg[i] = (d * Lcap + c * 8) * 2;
  }
  const int sw = hi ^ ((lo >> 3) & 1);
  const int k_frag = (lo >> 3) * KCG * 1024 + sw * 128 + (lo & 7) * 16;  // bytes
  const int v_frag = (lo >> 3) * 1024 + sw * 128 + (lo & 7) * 16;        // bytes
  const float lazy = 8.0f / sl2;

  {
    bf16x8 qf[D / 16];
    {
      const bf16* qrow = Q + ((long long)h * Mpad + q0 + lo) * D + hi * 8;
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16);
    }
    // staging sources: a wave-uniform per-head base plus 32-bit per-thread
    // byte offsets (the tile advance is a scalar add on the base)
    const char* Kh = reinterpret_cast<const char*>(Kc + (long long)h * Lcap * D);
    const char* Vh = reinterpret_cast<const char*>(Vt + (long long)h * D * Lcap);

    f32x16 oacc[DT];
#pragma unroll
    for (int i = 0; i < DT; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;

    auto dma_k = [&](int j, int buf) __attribute__((always_inline)) {
      const char* base = Kh + (long long)j * 64 * D * 2;
#pragma unroll
      for (int i = 0; i < KB; ++i)
        dma16(base + kg[i], (buf ? sK1 : sK0) + (wave + kWaves * i) * 512);
    };
    auto dma_v = [&](int j, int buf) __attribute__((always_inline)) {
      const char* base = Vh + (long long)j * 64 * 2;
#pragma unroll
      for (int i = 0; i < VB; ++i)
        dma16(base + vg[i], (buf ? sV1 : sV0) + (wave + kWaves * i) * 512);
    };
    auto qk = [&](f32x16* sacc, int buf) __attribute__((always_inline)) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[mt][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(reinterpret_cast<const char*>(buf ? sK1 : sK0) + k_frag +
                                                            mt * 4 * KCG * 1024 + (ks >> 2) * 1024 + (ks & 3) * 256);
          sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sacc[mt], 0, 0, 0);
        }
    };
    // keys past the window (last tile only) get -inf scores
    auto mask = [&](f32x16* sacc, int j) __attribute__((always_inline)) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = j * 64 + key_of_row(mt, (i >> 2) * 8 + hi * 4 + (i & 3));
          if (key >= Lk) sacc[mt][i] = -INFINITY;
        }
    };
    auto tile_max = [&](const f32x16* sacc) __attribute__((always_inline)) {
      float mx = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[mt][i]);
      return partner_max(mx);
    };
    // probabilities of one score tile against the settled running max m_run
    // (raw score units): p = 2^(s c - m c), c = log2(e)/sqrt(d)
    auto probs = [&](f32x16* sacc, bf16x8* pb) __attribute__((always_inline)) {
      const float msc = -m_run * sl2;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) sacc[mt][i] = __builtin_amdgcn_exp2f(fmaf(sacc[mt][i], sl2, msc));
#pragma unroll
      for (int kv = 0; kv < 4; ++kv)
#pragma unroll
        for (int i = 0; i < 8; ++i) pb[kv][i] = (bf16)sacc[kv >> 1][(kv & 1) * 8 + i];
      const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
      float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
      for (int kv = 0; kv < 4; ++kv) {
        ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[kv], pb[kv], 0, 1), ones, ps0, false);
        ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[kv], pb[kv], 2, 3), ones, ps1, false);
        ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[kv], pb[kv], 4, 5), ones, ps0, false);
        ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[kv], pb[kv], 6, 7), ones, ps1, false);
      }
      l_run += ps0 + ps1;
    };
    auto pv = [&](const bf16x8* pb, int buf) __attribute__((always_inline)) {
#pragma unroll
      for (int kv = 0; kv < 4; ++kv)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(reinterpret_cast<const char*>(buf ? sV1 : sV0) + v_frag +
                                                            dt * 4096 + kv * 256);
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[kv], oacc[dt], 0, 0, 0);
        }
    };
    // The running max moves only when a tile's max exceeds it by more than
    // 8/c (p then stays <= 2^8 in between, harmless for the float sums and
    // the bf16 probabilities); the rescale then also covers the tile just
    // added.
    auto update_max = [&](float mx) __attribute__((always_inline)) {
      if (mx > m_run + lazy) {
        const float alpha = __builtin_amdgcn_exp2f((m_run - mx) * sl2);
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
        m_run = mx;
      }
    };

    // prologue: K(k0), V(k0), K(k0+1) in LDS; S(k0) and its max
    dma_k(k0, 0);
    dma_v(k0, 0);
    if (k0 + 1 < k1) dma_k(k0 + 1, 1);
    XC_WAIT_VMCNT0();
    __syncthreads();
    if (!live) {
      __syncthreads();
      for (int j = k0; j < k1; ++j) {
        // the buffers iteration j of the compute loop refills
        const int odd = (j - k0) & 1;
        if (j + 2 < k1) dma_k(j + 2, odd);
        if (j + 1 < k1) dma_v(j + 1, 1 - odd);
        XC_WAIT_VMCNT0();
        __syncthreads();
      }
      return;
    }
    f32x16 sa[2], sb[2];
    qk(sa, 0);
    if (k0 == NT - 1) mask(sa, k0);
    m_run = tile_max(sa);
    __syncthreads();  // the first iteration refills K buffer 0, which S(k0) just read

    // Iteration j (local index jj = j - k0; scur = S(j), its max already in m_run):
    //   the DMA refills K(j+2) -> K buffer vb_cur and V(j+1) -> V buffer kb_next
    //   (both last read in iteration j - 1) are issued first and land during
    //   region 1: S(j+1) MFMAs from K buffer kb_next  ||  probabilities of S(j)
    //   region 2: PV(j) MFMAs from V buffer vb_cur     ||  max of S(j+1)
    //   then the (rare) rescale, the wait for this wave's DMA and the barrier.
    // The steady-state loop calls it with constant buffer arguments and no
    // mask: no branch inside.
    auto iter = [&](int j, f32x16* scur, f32x16* snext, int kb_next, int vb_cur, bool has_next, bool mask_next)
        __attribute__((always_inline)) {
      const bool more_k = j + 2 < k1;
      if (more_k) dma_k(j + 2, vb_cur);
      if (has_next) dma_v(j + 1, kb_next);
      if (has_next) qk(snext, kb_next);
      bf16x8 pb[4];
      probs(scur, pb);
      pv(pb, vb_cur);
      if (has_next) {
        if (mask_next) mask(snext, j + 1);
        update_max(tile_max(snext));
      }
      XC_WAIT_VMCNT0();
      __syncthreads();
    };
    const int n = k1 - k0;
    const int n_reg = n > 2 ? n - 2 : 0;  // iterations whose next tile is not the segment's last
    int jj = 0;
    for (; jj + 1 < n_reg; jj += 2) {
      iter(k0 + jj, sa, sb, 1, 0, true, false);
      iter(k0 + jj + 1, sb, sa, 0, 1, true, false);
    }
    if (jj < n_reg) {
      iter(k0 + jj, sa, sb, 1, 0, true, false);
      ++jj;
    }
    // the last two iterations: the next tile may be the masked global last
    // one, then there is no next tile
    const bool mask_last = (Lk & 63) != 0 && k1 == NT;
    if ((jj & 1) == 0) {
      if (jj + 1 < n) {
        iter(k0 + jj, sa, sb, 1, 0, true, mask_last);
        iter(k0 + jj + 1, sb, sa, 0, 1, false, false);
      } else {
        iter(k0 + jj, sa, sb, 1, 0, false, false);
      }
    } else {
      if (jj + 1 < n) {
        iter(k0 + jj, sb, sa, 0, 1, true, mask_last);
        iter(k0 + jj + 1, sa, sb, 1, 0, false, false);
      } else {
        iter(k0 + jj, sb, sa, 0, 1, false, false);
      }
    }

    const float l_tot = partner_sum(l_run);
    const int q = q0 + lo;
    if (n_split == 1) {
      // whole item in this unit: normalised output
      const float inv = 1.0f / l_tot;
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
    } else {
      // partial piece (see piece_floats)
      const int item = h * n_qt + qt;
      float* wo = ws + ((long long)item * n_split + kc) * piece_floats(D);
      bf16* wob = reinterpret_cast<bf16*>(wo);
      const int ql = wave * 32 + lo;
      const float inv = 1.0f / l_tot;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int dd = dt * 32 + g * 8 + hi * 4;
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          bf16x4 o4;
#pragma unroll
          for (int r = 0; r < 4; ++r) o4[r] = (bf16)(oacc[dt][g * 4 + r] * inv);
          *reinterpret_cast<bf16x4*>(wob + ql * D + dd) = o4;
        }
      if (hi == 0) {
        wo[kQT * D / 2 + ql] = m_run;
        wo[kQT * D / 2 + kQT + ql] = l_tot;
      }
    }
  }
}

// Combines the S pieces of each item in a fixed order (deterministic):
// O = sum_p w_p l_p Ohat_p / sum_p w_p l_p, w_p = 2^((m_p - M) c),
// M = max_p m_p, Ohat_p the piece's normalised output.
// One workgroup per 32 queries of an item; a thread owns one query and 16
// consecutive head dims.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(bf16* __restrict__ O, int L, int H, int n_qt, int n_split,
                                                         float sl2, const float* __restrict__ ws,
                                                         const int* __restrict__ flag) {
  if (flag != nullptr && *flag) return;
  constexpr int TPQ = D / 16;  // threads per query
  constexpr int QPB = 256 / TPQ;  // queries per workgroup
  const int blocks_per_item = kQT / QPB;
  const int item = blockIdx.x / blocks_per_item;
  const int ql = (blockIdx.x % blocks_per_item) * QPB + threadIdx.x / TPQ;
  const int d0 = (threadIdx.x % TPQ) * 16;
  const int h = item / n_qt, qt = item - h * n_qt;
  const int q = qt * kQT + ql;
  if (q >= L) return;
  const long long stride = piece_floats(D);
  const float* base = ws + (long long)item * n_split * stride;
  float M = -INFINITY;
  for (int p = 0; p < n_split; ++p) M = fmaxf(M, base[p * stride + kQT * D / 2 + ql]);
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  float den = 0.f;
  for (int p = 0; p < n_split; ++p) {
    const float* pp = base + p * stride;
    const float w = __builtin_amdgcn_exp2f((pp[kQT * D / 2 + ql] - M) * sl2) * pp[kQT * D / 2 + kQT + ql];
    den += w;
    const bf16x8* src = reinterpret_cast<const bf16x8*>(reinterpret_cast<const bf16*>(pp) + ql * D + d0);
    const bf16x8 v0 = src[0], v1 = src[1];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      acc[i] += w * (float)v0[i];
      acc[8 + i] += w * (float)v1[i];
    }
  }
  const float inv = 1.0f / den;
  bf16x8 o0, o1;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    o0[i] = (bf16)(acc[i] * inv);
    o1[i] = (bf16)(acc[8 + i] * inv);
  }
  bf16* orow = O + (long long)q * H * D + h * D + d0;
  *reinterpret_cast<bf16x8*>(orow) = o0;
  *reinterpret_cast<bf16x8*>(orow + 8) = o1;
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

int resident_attention_groups() {
  static int groups[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 512;
  if (groups[dev] == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
    groups[dev] = cus;
  }
  return groups[dev];
}

// Key splits per item.  Estimated time in key-tile steps of one resident
// workgroup: rounds * (tiles per unit + 4 for the unit's prologue and
// epilogue) + 4 S items / (resident workgroups) for the merge (fitted to
// measured split sweeps on the multi-camera shapes, where it picks S = 3),
// over S <= 16 with chunks of at least 4 tiles: few items over a long window
// (768 tokens, 8 heads, 3072 keys: 24 items) take more splits; only split
// counts whose partials fit in cap_floats workspace floats are considered
// (S = 1 needs none).
int attention_splits(int L, int Lk, int H, int D, size_t cap_floats) {
  const int items = H * ((L + kQT - 1) / kQT);
  const int NT = (Lk + 63) / 64;
  const int slots = resident_attention_groups();
  int best = 1;
  double best_cost = 1e300;
  for (int s = 1; s <= 16 && (s == 1 || NT / s >= 4); ++s) {
    if (s > 1 && (size_t)items * s * (size_t)piece_floats(D) > cap_floats) break;
    const long long units = (long long)items * s;
    const long long rounds = (units + slots - 1) / slots;
    const double cost = (double)rounds * ((double)NT / s + 4.0) + (s > 1 ? 4.0 * s * items / slots : 0.0);
    if (cost < best_cost - 1e-9) {
      best_cost = cost;
      best = s;
    }
  }
  return best;
}

size_t attention_workspace_floats(int L, int Lk, int H, int D) {
  const int s = attention_splits(L, Lk, H, D, SIZE_MAX);
  if (s == 1) return 0;
  return (size_t)H * ((L + kQT - 1) / kQT) * s * (size_t)piece_floats(D);
}

// bf16 requirements (checked by the caller): D in {64, 128}; Q has Mpad >=
// roundup(L, 256) rows per head; the caches have Lcap >= roundup(Lk, 64) rows,
// Lcap a multiple of 8 (16-byte aligned V^T rows for the DMA), 16-byte
// aligned bases, and keys past Lk that hold finite values; ws holds ws_floats floats (the key
// split is limited to what fits: attention_workspace_floats(L, Lk, H, D)
// floats allow the unconstrained choice).
void launch_attention(int dtype, const void* q, const void* kc, const void* vt, void* o, float* ws, size_t ws_floats,
                      int L, int Mpad, int Lcap, int Lk, int H, int D, const int* flag, hipStream_t st) {
  if (dtype == 1) {
    const int n_qt = (L + kQT - 1) / kQT;
    const int n_split = attention_splits(L, Lk, H, D, ws != nullptr ? ws_floats : 0);
    const int units = H * n_split * n_qt;
    const int grid = (units + kXcds - 1) / kXcds * kXcds;
    const float sl2 = 1.4426950408889634f / sqrtf((float)D);
    const int merge_grid = H * n_qt * (kQT / (256 / (D / 16)));
    if (D == 128) {
      attn_bf16_kernel<128><<<grid, 64 * kWaves, 0, st>>>((const bf16*)q, (const bf16*)kc, (const bf16*)vt, (bf16*)o, L,
                                                  Mpad, Lcap, Lk, H, n_qt, n_split, sl2, ws, flag);
      if (n_split > 1) attn_merge_kernel<128><<<merge_grid, 256, 0, st>>>((bf16*)o, L, H, n_qt, n_split, sl2, ws, flag);
    } else {
      attn_bf16_kernel<64><<<grid, 64 * kWaves, 0, st>>>((const bf16*)q, (const bf16*)kc, (const bf16*)vt, (bf16*)o, L,
                                                 Mpad, Lcap, Lk, H, n_qt, n_split, sl2, ws, flag);
      if (n_split > 1) attn_merge_kernel<64><<<merge_grid, 256, 0, st>>>((bf16*)o, L, H, n_qt, n_split, sl2, ws, flag);
    }
  } else {
    dim3 grid(L, H);
    attn_f32_kernel<<<grid, 64, 0, st>>>((const float*)q, (const float*)kc, (const float*)vt, (float*)o, L, Mpad,
                                         Lcap, Lk, H, D, 1.0f / sqrtf((float)D), flag);
  }
}

}  // namespace xc
